"""GPU (HIP library, through the C ABI) vs the CPU oracle, element by element.

Bit-exact for every block key, matched-prefix length, target, branch and the sorted
index dump.  Sizes keep the oracle at seconds while spanning several 64-block tiles,
ragged tails, shared prefixes held by more instances than a holder list keeps (bitmap
records), pool exhaustion, eviction with orphaned descendants, and the degenerate cases
(empty prompts, empty batches, one instance)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_08565_amd import workload as W
from tests.parity import Pair, run_sessions, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _rand_prompts(rng, n, lo, hi, vocab=W.VOCAB):
    lens = rng.integers(lo, hi, n)
    toks = rng.integers(0, vocab, int(lens.sum()), dtype=np.int32)
    off = np.zeros(n + 1, np.int64)
    off[1:] = np.cumsum(lens)
    return toks, off


@pytest.mark.parametrize("B", [16, 2, 8, 32, 256])
def test_hash_parity_ragged(B):
    rng = np.random.default_rng(B)
    toks, off = _rand_prompts(rng, 37, 0, 5000)
    # extremes: empty, one token short of a block, exactly one block, a multi-tile prompt
    extra = [0, B - 1, B, 64 * B * 3 + B * 5 + 3]
    for L in extra:
        toks = np.concatenate([toks, rng.integers(-2**31, 2**31 - 1, L, dtype=np.int64).astype(np.int32)])
        off = np.append(off, off[-1] + L)
    pair = Pair(1024, 4, seed=int(rng.integers(0, 2**63)), block=B)
    say(f"hash B={B} blocks={int((np.diff(off) // B).sum())}")
    pair.hash_both(toks, off)


def test_hash_long_prompt_many_tiles():
    rng = np.random.default_rng(1)
    toks, off = _rand_prompts(rng, 3, 131072 - 7, 131072 + 1)
    Pair(16, 1).hash_both(toks, off)


def test_hash_bad_offsets_flag_status_without_writing():
    from paper_2607_08565_amd import smetric as S
    toks = to_dev(np.arange(64, dtype=np.int32))
    tok_off = to_dev(np.array([0, 32, 64], np.int64))
    blk_off = to_dev(np.array([0, 3, 5], np.int64))  # request 0 claims 3 blocks of a 2-block prompt
    keys = to_dev(np.full(5, 7, np.uint64))
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    S.hash_blocks(toks, tok_off, blk_off, 5, 16, 5, keys=keys, status=status)
    got = keys.cpu().numpy()
    assert int(status.item()) == S.EINVAL
    assert got[:3].tolist() == [7, 7, 7]  # the bad request wrote nothing
    _, ok = oracle.hash_blocks(np.arange(64, dtype=np.int32)[32:], [0, 32], 16, 5)
    assert got[3:].tolist() == ok.tolist()  # the good one is unaffected


@pytest.mark.parametrize("probed", [False, True])
def test_config0_open_loop_full(probed):
    """The tiny trace at full size: 8 instances, 64 sessions x 4 turns."""
    pair, br = run_sessions(W.config0(), 4, capacity=200_000, probed=probed)
    assert set(br.tolist()) >= {0, 2}


@pytest.mark.parametrize("probed", [False, True])
def test_config1_scaled_closed_loop(probed):
    wl = W.config1(n_sess=192, n_turns=8, l0=1024, app=(64, 1536), cap=16384, prefix_len=512)
    pair, br = run_sessions(wl, 8, capacity=2_000_000, probed=probed)
    say("branches", np.bincount(br, minlength=5).tolist())


@pytest.mark.parametrize("probed", [False, True])
def test_config2_scaled_prev_counts(probed):
    wl = W.config2(n_sess=48, n_turns=10, l0=4096, app=(128, 3000), cap=40000, prefix_len=2048)
    run_sessions(wl, 10, capacity=2_000_000, probed=probed)


@pytest.mark.parametrize("probed", [False, True])
@pytest.mark.parametrize("frac", [(1, 20), (1, 3)])
def test_config3_scaled_with_eviction(probed, frac):
    """One shared prefix held by every instance (bitmap records, WIDE alive sets of 128),
    divergent tails, LRU eviction after every batch (orphaned descendants).  5 % per batch
    evicts in place (tombstones, members leaving their bitmaps); a third per batch passes
    the tombstone limit and rebuilds the table."""
    wl = W.config3(n_sess=160, n_turns=5, prefix_len=4096, tail=(256, 3000), app=512)
    run_sessions(wl, 5, capacity=400_000, evict=frac, probed=probed)


def test_config3_tombstones_accumulate_then_rebuild():
    """An eighth evicted after each of ten batches: the first evictions leave tombstones in
    place (inserts, matches and later evictions run over them), then the tombstones pass
    the limit and the table is rebuilt; the dump equals the oracle's after every step."""
    wl = W.config3(n_sess=160, n_turns=10, prefix_len=4096, tail=(256, 3000), app=512)
    run_sessions(wl, 10, capacity=400_000, evict=(1, 8), probed=True)


def test_partition_overlaps_previous_insert():
    """Two streams: batch t+1's hash and partition run while batch t's insert is still
    queued on the other stream (the partition reads the index geometry only); lookup waits
    for both.  Every matched row, target, branch and the final dump equal the oracle's."""
    from paper_2607_08565_amd import smetric as S
    wl = W.config1(n_sess=192, n_turns=6, l0=1024, app=(64, 1536), cap=16384, prefix_len=512)
    pair = Pair(2_000_000, wl.n_inst)
    sA, sB = torch.cuda.Stream(), torch.cuda.Stream()
    keys = [torch.empty(1 << 20, dtype=torch.uint64, device="cuda") for _ in range(2)]
    states = [None, None]
    prev_t, held = None, []
    for t in range(6):
        b = wl.batch(t, prev_t)
        blk_off, nb = S.block_offsets(b.tok_off)
        assert nb <= keys[0].numel()
        d_tok, d_toff, d_boff = to_dev(b.tokens), to_dev(b.tok_off), to_dev(blk_off)
        held.append((d_tok, d_toff, d_boff))  # read on other streams: keep them alive to the end
        p = t % 2
        # keys[p] and states[p] were last read by batch t-2, finished at t-1's synchronize below
        sA.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(sA):
            S.hash_blocks(d_tok, d_toff, d_boff, nb, keys=keys[p])
            states[p] = pair.gix.probe_partition(keys[p], d_boff, nb, state=states[p])
            front = torch.cuda.Event()
            front.record(sA)
        _, okeys = oracle.hash_blocks(b.tokens, b.tok_off, W.BLOCK, W.DEFAULT_SEED)
        with torch.cuda.stream(sB):
            sB.wait_event(front)
            pair.gix.probe_lookup(states[p], keys[p], d_boff, nb)
            gm = pair.gix.match_probed(states[p], keys[p], d_boff, nb)
            gt, gb = S.route(gm, to_dev(b.prompt_len), to_dev(b.hist_len), to_dev(b.turn), to_dev(b.q),
                             W.DEFAULT_PARAMS, b.rr_base)
            sB.synchronize()
            om = pair.oix.match(okeys, blk_off)
            ot, ob = oracle.route(om, b.prompt_len, b.hist_len, b.turn, b.q, W.DEFAULT_PARAMS, b.rr_base)
            assert np.array_equal(gm.cpu().numpy(), om), f"batch {t}: matched rows differ"
            assert np.array_equal(gt.cpu().numpy(), ot) and np.array_equal(gb.cpu().numpy(), ob), f"batch {t}"
            # the insert stays queued on sB while the loop builds, hashes and partitions t+1 on sA
            pair.gix.insert_probed(states[p], b.n_req, nb, to_dev(np.asarray(ot, np.int32)),
                                   to_dev(np.asarray(b.session, np.uint32)), b.epoch)
        assert pair.oix.insert(okeys, blk_off, ot, b.session, b.epoch) == 0
        prev_t = ot
        say(f"  batch {t}: R={b.n_req} blocks={nb}")
    torch.cuda.synchronize()
    pair.compare_index("after the pipelined batches")


def test_many_instances_wide_words():
    """I = 5000 (two bitmap words per lane) and a prefix shared by 300 instances."""
    rng = np.random.default_rng(5)
    I = 5000
    pre = rng.integers(0, W.VOCAB, 2048, dtype=np.int32)
    pair = Pair(2_000_000, I)
    prompts = [np.concatenate([pre[: rng.integers(100, 2048)], rng.integers(0, W.VOCAB, rng.integers(0, 900), dtype=np.int32)])
               for _ in range(300)]
    off = np.zeros(301, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    toks = np.concatenate(prompts)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)
    inst = rng.choice(I, 300, replace=False).astype(np.int32)
    assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, inst, np.arange(300), 1) == 0
    pair.compare_index("insert")
    q = np.concatenate([pre, rng.integers(0, W.VOCAB, 500, dtype=np.int32)])
    batch = W.Batch(tokens=np.concatenate([q, q[:1000]]), tok_off=np.array([0, len(q), len(q) + 1000]),
                    prompt_len=np.array([len(q), 1000], np.int32), hist_len=np.array([1024, 0], np.int32),
                    turn=np.array([1, 0], np.int32), session=np.array([9, 10], np.uint32),
                    q=rng.integers(0, 50, I) * W.Q_UNIT_NS, rr_base=17, epoch=2)
    pair.step(batch, what="I=5000")
    pair.step(batch, what="I=5000 probed", probed=True)


@pytest.mark.parametrize("I", [130, 300, 1000, 4000])
def test_wide_mode_bitmap_widths(I):
    """Bitmap rows of 3, 5, 16 and 63 words (lane groups of 4, 8, 16 and 64 lanes, the odd
    widths with padding lanes): a prefix held by most instances to different depths, so the
    alive set shrinks block by block through the wide mode and hands over to the narrow
    one; many requests, each probing the prefix to its own length."""
    rng = np.random.default_rng(I)
    pre = rng.integers(0, W.VOCAB, 4096, dtype=np.int32)
    pair = Pair(3_000_000, I)
    n_hold = int(0.8 * I)
    prompts = [np.concatenate([pre[: rng.integers(64, 4096)], rng.integers(0, W.VOCAB, rng.integers(0, 600), dtype=np.int32)])
               for _ in range(n_hold)]
    off = np.zeros(n_hold + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(np.concatenate(prompts), off)
    inst = rng.choice(I, n_hold, replace=False).astype(np.int32)
    assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, inst, np.arange(n_hold), 1) == 0
    R = 48
    qs = [np.concatenate([pre[: rng.integers(16, 4096)], rng.integers(0, W.VOCAB, rng.integers(0, 2000), dtype=np.int32)])
          for _ in range(R)]
    toff = np.zeros(R + 1, np.int64)
    toff[1:] = np.cumsum([len(x) for x in qs])
    batch = W.Batch(tokens=np.concatenate(qs), tok_off=toff, prompt_len=np.diff(toff).astype(np.int32),
                    hist_len=rng.integers(0, 4096, R).astype(np.int32), turn=rng.integers(0, 3, R).astype(np.int32),
                    session=np.arange(R, dtype=np.uint32) + 5000, q=rng.integers(0, 50, I) * W.Q_UNIT_NS,
                    rr_base=3, epoch=2)
    say(f"I={I}: {n_hold} holders, {nb} blocks inserted")
    pair.step(batch, what=f"I={I}", check_dump=False)
    pair.step(batch, what=f"I={I} probed", probed=True)


def test_max_instances():
    rng = np.random.default_rng(6)
    I = 65536
    pre = rng.integers(0, W.VOCAB, 512, dtype=np.int32)
    pair = Pair(200_000, I)
    R = 80
    prompts = [np.concatenate([pre, rng.integers(0, W.VOCAB, 100, dtype=np.int32)]) for _ in range(R)]
    off = np.zeros(R + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(np.concatenate(prompts), off)
    inst = np.concatenate([rng.choice(I, R - 2, replace=False), [0, I - 1]]).astype(np.int32)
    assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, inst, np.arange(R), 3) == 0
    pair.compare_index("insert")
    b = W.Batch(tokens=prompts[0][:600], tok_off=np.array([0, 600]), prompt_len=np.array([600], np.int32),
                hist_len=np.array([512], np.int32), turn=np.array([1], np.int32), session=np.array([1], np.uint32),
                q=np.zeros(I, np.int64), rr_base=0, epoch=4)
    pair.step(b, what="I=65536")
    pair.step(b, what="I=65536 probed", probed=True)


def test_hot_keys_pool_exhaustion_and_long_lists():
    """More hot keys than bitmap records: the rest keep long plain holder lists."""
    rng = np.random.default_rng(7)
    I, R = 16, 12 * 16
    pair = Pair(40_000, I)  # 156 bitmap records for ~1,800 keys held by all 16 instances
    streams = [rng.integers(0, W.VOCAB, 16 * 150, dtype=np.int32) for _ in range(12)]
    prompts = [streams[r % 12][: 16 * rng.integers(100, 150)] for r in range(R)]
    off = np.zeros(R + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(np.concatenate(prompts), off)
    inst = np.array([r // 12 for r in range(R)], np.int32)  # each stream on all 16 instances
    assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, inst, np.arange(R), 1) == 0
    pair.compare_index("insert")
    b = W.Batch(tokens=np.concatenate(streams[:4]), tok_off=np.arange(5) * 16 * 150,
                prompt_len=np.full(4, 2400, np.int32), hist_len=np.full(4, 1600, np.int32),
                turn=np.ones(4, np.int32), session=np.arange(4, dtype=np.uint32), q=np.zeros(I, np.int64), epoch=2)
    pair.step(b, what="hot")
    pair.step(b, what="hot probed", probed=True)


def test_duplicate_pairs_in_batch_take_lowest_request():
    rng = np.random.default_rng(8)
    pair = Pair(10_000, 4)
    p = rng.integers(0, W.VOCAB, 800, dtype=np.int32)
    prompts = [p[:800], p[:400], p[:800], p[:640]]
    off = np.zeros(5, np.int64)
    off[1:] = np.cumsum([len(x) for x in prompts])
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(np.concatenate(prompts), off)
    assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, [2, 2, 2, 1], [50, 40, 30, 20], 5) == 0
    pair.compare_index("dups")
    assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, [2, 3, 2, 1], [9, 8, 7, 6], 3) == 0
    pair.compare_index("older epoch")


def test_efull_and_einval_leave_index_unchanged():
    rng = np.random.default_rng(9)
    pair = Pair(100, 3)
    toks, off = _rand_prompts(rng, 4, 300, 700)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)
    half = np.array([0, nb // 2])
    rc = pair.insert_both(d_keys, to_dev(half), nb, okeys, half, [1], [1], 1)
    assert rc == 0
    pair.compare_index("first")
    rc = pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, [0, 1, 2, 0], [1, 2, 3, 4], 2)
    assert rc == oracle.EFULL
    pair.compare_index("efull")
    # instance out of range -> EINVAL, unchanged (status stays the first error: EFULL)
    rc = pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, [0, 5, 1, 1], [1, 2, 3, 4], 3)
    assert rc == oracle.EINVAL
    pair.compare_index("einval")
    _, st = pair.gix.stats(reset_status=True)
    assert st == oracle.EFULL and pair.gix.stats()[1] == 0


def _probed_insert_both(pair, d_keys, d_boff, nb, okeys, blk_off, inst, sess, epoch):
    """The region-ordered insert (probe state -> insert) on the GPU, the oracle's insert on the CPU."""
    n_req = len(blk_off) - 1
    state = pair.gix.probe(d_keys, d_boff, nb)
    pair.gix.insert_probed(state, n_req, nb, to_dev(np.asarray(inst, np.int32)), to_dev(np.asarray(sess, np.uint32)),
                           epoch)
    return pair.oix.insert(okeys, blk_off, inst, sess, epoch)


def test_probed_insert_oversized_bins_and_duplicates():
    """Thousands of candidates of the same few keys: their bins exceed the LDS pair table and
    go through the fallback pair table; repeated (key, instance) pairs keep the lowest request."""
    rng = np.random.default_rng(21)
    I, R = 512, 4096
    pair = Pair(400_000, I)
    base = rng.integers(0, W.VOCAB, 16 * 40, dtype=np.int32)
    prompts = [base[: 16 * int(rng.integers(20, 41))] for _ in range(R)]
    off = np.zeros(R + 1, np.int64)
    off[1:] = np.cumsum([len(x) for x in prompts])
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(np.concatenate(prompts), off)
    say(f"oversized bins: {nb} candidates of 40 keys")
    inst = rng.integers(0, I, R).astype(np.int32)
    sess = rng.permutation(R).astype(np.uint32)  # lowest request != lowest session
    assert _probed_insert_both(pair, d_keys, d_boff, nb, okeys, blk_off, inst, sess, 3) == 0
    pair.compare_index("oversized bins")
    # again with new instances and an older epoch: refreshes keep the newer epoch
    inst2 = rng.integers(0, I, R).astype(np.int32)
    assert _probed_insert_both(pair, d_keys, d_boff, nb, okeys, blk_off, inst2, sess[::-1].copy(), 2) == 0
    pair.compare_index("oversized bins, second batch")


def test_probed_insert_errors_and_two_pass_refresh():
    """The region-ordered insert's all-or-nothing errors, and its refresh pass when an error
    cannot be ruled out beforehand (the index near capacity, or an invalid request without blocks)."""
    rng = np.random.default_rng(22)
    pair = Pair(100, 3)
    toks, off = _rand_prompts(rng, 4, 300, 700)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)
    half = np.array([0, nb // 2])
    assert _probed_insert_both(pair, d_keys, to_dev(half), nb // 2, okeys, half, [1], [1], 1) == 0
    pair.compare_index("first")
    assert _probed_insert_both(pair, d_keys, d_boff, nb, okeys, blk_off, [0, 1, 2, 0], [1, 2, 3, 4], 2) == oracle.EFULL
    pair.compare_index("efull")
    assert _probed_insert_both(pair, d_keys, d_boff, nb, okeys, blk_off, [0, 5, 1, 1], [1, 2, 3, 4], 3) == oracle.EINVAL
    pair.compare_index("einval")
    _, st = pair.gix.stats(reset_status=True)
    assert st == oracle.EFULL and pair.gix.stats()[1] == 0
    # entries + blocks > capacity, but the new pairs fit: refreshes in their own pass
    near = Pair(100, 3)
    near.hash_both(toks, off)
    assert _probed_insert_both(near, d_keys, to_dev(half), nb // 2, okeys, half, [1], [1], 1) == 0
    assert near.oix.size + nb // 2 > 100
    assert _probed_insert_both(near, d_keys, to_dev(half), nb // 2, okeys, half, [1], [7], 4) == 0
    near.compare_index("refresh pass near capacity")
    # a request without blocks may name any target; the others' pairs are entered
    big = Pair(10_000, 3)
    off2 = np.concatenate([off[:2], off[1:2], off[2:] - 0])  # request 1 is empty
    toks2 = toks
    d_boff2, nb2, d_keys2, okeys2, blk_off2 = big.hash_both(toks2, off2)
    assert _probed_insert_both(big, d_keys2, d_boff2, nb2, okeys2, blk_off2, [0, 9, 1, 2, 0], [1, 2, 3, 4, 5], 1) == 0
    big.compare_index("empty request with an invalid target")
    assert _probed_insert_both(big, d_keys2, d_boff2, nb2, okeys2, blk_off2, [2, 9, 1, 0, 0], [6, 7, 8, 9, 10], 2) == 0
    big.compare_index("refresh pass after an invalid empty request")


@pytest.mark.parametrize("B", [16, 8])
def test_hash_partition_equals_the_separate_calls(B):
    """smetric_hash_partition (the hash taking the partition's region counts itself for
    B = 16) leaves the same keys and probe state as hash + partition: every block key,
    matched row, decision and the index after the insert equal the oracle's."""
    rng = np.random.default_rng(30 + B)
    I = 64
    pair = Pair(2_000_000, I, block=B)
    pre = rng.integers(0, W.VOCAB, 64 * B * 3, dtype=np.int32)
    prompts = [np.concatenate([pre[: int(rng.integers(0, len(pre)))],
                               rng.integers(0, W.VOCAB, int(rng.integers(0, 70 * B)), dtype=np.int32)])
               for _ in range(300)]
    off = np.zeros(301, np.int64)
    off[1:] = np.cumsum([len(x) for x in prompts])
    toks = np.concatenate(prompts)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)  # warm the index with half of them
    half = 150
    hb = blk_off[: half + 1]
    assert pair.insert_both(d_keys, to_dev(hb), int(hb[-1]), okeys, hb, rng.integers(0, I, half).astype(np.int32),
                            np.arange(half), 1) == 0
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    keys, state = pair.gix.hash_partition(to_dev(toks), to_dev(off), d_boff, nb, block_size=B, seed=pair.seed,
                                          status=status)
    assert int(status.item()) == 0
    assert np.array_equal(keys[:nb].cpu().numpy(), okeys), "keys"
    pair.gix.probe_lookup(state, keys, d_boff, nb)
    gm = pair.gix.match_probed(state, keys, d_boff, nb).cpu().numpy()
    om = pair.oix.match(okeys, blk_off)
    assert np.array_equal(gm, om), "matched rows"
    R = len(prompts)
    inst = rng.integers(0, I, R).astype(np.int32)
    pair.gix.insert_probed(state, R, nb, to_dev(inst), to_dev(np.arange(R, dtype=np.uint32) + 500), 2)
    assert pair.oix.insert(okeys, blk_off, inst, np.arange(R) + 500, 2) == 0
    pair.compare_index(f"hash_partition B={B}")


def test_hash_partition_bad_token_range_invalidates_the_state():
    """A request whose token range does not give its block count: the hash flags status,
    the counting hash marks the probe state invalid, and the consumers report EINVAL
    without touching anything out of bounds."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(33)
    pair = Pair(10_000, 4)
    toks = rng.integers(0, W.VOCAB, 16 * 40, dtype=np.int32)
    tok_off = np.array([0, 16 * 10, 16 * 25, 16 * 40], np.int64)
    blk_off = np.array([0, 10, 27, 40], np.int64)  # request 1 claims 17 blocks of a 15-block range
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    d_boff = to_dev(blk_off)
    keys, state = pair.gix.hash_partition(to_dev(toks), to_dev(tok_off), d_boff, 40, status=status)
    assert int(status.item()) == S.EINVAL
    pair.gix.probe_lookup(state, keys, d_boff, 40)
    m = pair.gix.match_probed(state, keys, d_boff, 40).cpu().numpy()
    assert not m.any()
    _, st = pair.gix.stats(reset_status=True)
    assert st == S.EINVAL
    pair.gix.insert_probed(state, 3, 40, to_dev(np.array([0, 1, 2], np.int32)), to_dev(np.array([1, 2, 3], np.uint32)), 1)
    n, st = pair.gix.stats()
    assert n == 0 and st == S.EINVAL


def test_hash_partition_with_no_full_block():
    """Every prompt shorter than one block: no keys, an empty probe state, all-zero matched
    rows, nothing inserted and no error, on the fused call's counting path."""
    rng = np.random.default_rng(34)
    pair = Pair(10_000, 6)
    lens = np.array([0, 1, 15, 7, 0, 15], np.int64)
    tok_off = np.zeros(len(lens) + 1, np.int64)
    tok_off[1:] = np.cumsum(lens)
    toks = rng.integers(0, W.VOCAB, int(tok_off[-1]), dtype=np.int32)
    blk_off = np.zeros(len(lens) + 1, np.int64)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    d_boff = to_dev(blk_off)
    keys, state = pair.gix.hash_partition(to_dev(toks), to_dev(tok_off), d_boff, 0, status=status)
    assert int(status.item()) == 0
    pair.gix.probe_lookup(state, keys, d_boff, 0)
    m = pair.gix.match_probed(state, keys, d_boff, 0).cpu().numpy()
    assert m.shape == (len(lens), 6) and not m.any()
    R = len(lens)
    pair.gix.insert_probed(state, R, 0, to_dev(np.zeros(R, np.int32)), to_dev(np.arange(R, dtype=np.uint32)), 1)
    assert pair.gix.stats() == (0, 0)


def test_match_bad_range_and_empty_requests():
    rng = np.random.default_rng(10)
    pair = Pair(10_000, 5)
    toks, off = _rand_prompts(rng, 3, 200, 400)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)
    pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, [0, 1, 2], [1, 2, 3], 1)
    bad = np.array([0, blk_off[1], blk_off[1] - 1, nb, nb], np.int64)  # request 1 decreasing, 3 empty
    gm = pair.gix.match(d_keys, to_dev(bad), nb).cpu().numpy()
    om = pair.oix.match(okeys, bad, nb)
    assert np.array_equal(gm, om)
    assert pair.gix.stats()[1] == oracle.EINVAL == pair.oix.status


def test_evict_everything_then_refill():
    """Evicting all entries leaves only tombstones (in place), the next batch is matched
    against an empty index and inserted over them, nothing-to-evict is a no-op, and a
    second full eviction rebuilds; the dump equals the oracle's after every step."""
    rng = np.random.default_rng(77)
    pair = Pair(2_000, 6)  # small: the third full eviction passes the tombstone limit
    for step in range(3):
        toks, off = _rand_prompts(rng, 12, 200, 900)
        d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)
        gm = pair.gix.match(d_keys, d_boff, nb).cpu().numpy()
        assert np.array_equal(gm, pair.oix.match(okeys, blk_off)), f"step {step}: matched rows"
        inst = rng.integers(0, 6, 12).astype(np.int32)
        assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, inst, np.arange(12) + 100 * step, step + 1) == 0
        pair.compare_index(f"step {step} insert")
        pair.gix.evict(0, 5)
        assert pair.oix.evict(0, 5) == 0
        pair.compare_index(f"step {step} evict nothing")
        if step != 1:
            pair.gix.evict(1, 1)
            assert pair.oix.evict(1, 1) == 0
            pair.compare_index(f"step {step} evict everything")
            assert pair.gix.stats()[0] == 0


def test_empty_batch_and_single_instance():
    from paper_2607_08565_amd import smetric as S
    pair = Pair(1000, 1)
    b = W.Batch(tokens=np.zeros(0, np.int32), tok_off=np.zeros(1, np.int64), prompt_len=np.zeros(0, np.int32),
                hist_len=np.zeros(0, np.int32), turn=np.zeros(0, np.int32), session=np.zeros(0, np.uint32),
                q=np.zeros(1, np.int64))
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(b.tokens, b.tok_off)
    assert nb == 0
    rng = np.random.default_rng(11)
    toks, off = _rand_prompts(rng, 5, 0, 100)
    b = W.Batch(tokens=toks, tok_off=off, prompt_len=np.diff(off).astype(np.int32), hist_len=np.zeros(5, np.int32),
                turn=np.array([0, 1, 2, 0, 1], np.int32), session=np.arange(5, dtype=np.uint32), q=np.array([7], np.int64))
    pair.step(b, what="I=1 a")
    pair.step(b, what="I=1 b")
    pair.step(b, what="I=1 c", probed=True)
    assert S.version() >= 1


def test_route_edge_parameters():
    """SLACK = inf / 0, HIT_RATIO 0, c_att = 0, and out-of-domain requests (branch 255)."""
    rng = np.random.default_rng(12)
    R, I = 300, 40
    m = rng.integers(0, 60, (R, I)).astype(np.int32)
    L = rng.integers(0, 1200, R).astype(np.int32)
    m = np.minimum(m, (L // 16)[:, None]).astype(np.int32)
    m[5, 3] = -1
    m[6, 0] = L[6] // 16 + 1
    hist = rng.integers(0, 1200, R).astype(np.int32)
    hist[7] = -1
    turn = rng.integers(0, 3, R).astype(np.int32)
    turn[8] = -2
    L[9] = -5
    q = rng.integers(0, 200, I).astype(np.int64) * W.Q_UNIT_NS
    from paper_2607_08565_amd import smetric as S
    for over in ({}, dict(slack_num=0, slack_den=0), dict(slack_num=0, slack_den=1), dict(hit_num=0, hit_den=7),
                 dict(c_att=0, c_lin=1), dict(slack_num=3, slack_den=2, c_att=4)):
        p = dict(W.DEFAULT_PARAMS, **over)
        for rr in (0, 123456789):
            gt, gb = S.route(to_dev(m), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q), p, rr)
            ot, ob = oracle.route(m, L, hist, turn, q, p, rr)
            assert np.array_equal(gt.cpu().numpy(), ot) and np.array_equal(gb.cpu().numpy(), ob), over
    assert set(ob[[5, 6, 7, 8, 9]].tolist()) == {255}
    with pytest.raises(S.SmetricError):
        S.route(to_dev(m), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q), dict(W.DEFAULT_PARAMS, hit_num=2, hit_den=2))


def test_route_scan_precision_boundaries():
    """The route scans in doubles while C0 = 2 C_LIN L + C_ATT L^2 and every 2q stay below
    2^50 (each score is then an integer below 2^51) and in 128 bits otherwise: prompts whose
    C0 falls just under and at 2^50 (C_ATT = C_LIN = 2^32, L around 511-512), queues just
    under and at 2^49 on some instances, exact ties between instances, and wavefronts that
    switch to 128 bits with an out-of-domain request among them."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(14)
    big = dict(W.DEFAULT_PARAMS, c_lin=1 << 32, c_att=1 << 32, slo_b=1 << 32, slo_a=1 << 32,
               slack_num=1 << 20, slack_den=1, block_size=16)
    for I in (1, 37, 64, 65, 1024, 1500):
        R = 400
        L = rng.integers(500, 520, R).astype(np.int32)
        m = rng.integers(0, 33, (R, I))
        m = np.minimum(m, (L // 16)[:, None]).astype(np.int32)
        m[:, ::3] = m[:, :1]  # ties on c, so ties on the scores
        hist = rng.integers(0, 520, R).astype(np.int32)
        turn = rng.integers(0, 3, R).astype(np.int32)
        for qcase in range(4):
            if qcase == 0:    # all far below 2^49
                q = rng.integers(0, 1 << 30, I)
            elif qcase == 1:  # up to 2^49 - 1: the double scan
                q = rng.integers((1 << 49) - 4096, 1 << 49, I)
            elif qcase == 2:  # one instance at 2^49: the 128-bit scan
                q = rng.integers((1 << 49) - 4096, 1 << 49, I)
                q[rng.integers(0, I)] = 1 << 49
            else:             # equal queues, every tie down to the rotation
                q = np.full(I, (1 << 49) - 1)
            q = q.astype(np.int64)
            for p in (big, dict(big, c_att=(1 << 32) - 1), dict(big, c_lin=0), W.DEFAULT_PARAMS):
                m2 = m.copy()
                m2[7, 0] = 1 << 20  # an out-of-domain request
                for rr in (0, 2**64 - 1):
                    gt, gb = S.route(to_dev(m2), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q), p, rr)
                    ot, ob = oracle.route(m2, L, hist, turn, q, p, rr)
                    assert np.array_equal(gt.cpu().numpy(), ot) and np.array_equal(gb.cpu().numpy(), ob), \
                        (I, qcase, p["c_lin"], p["c_att"], rr)
                assert ob[7] == 255


def test_probed_path_rejects_untiled_requests():
    """The region-ordered path needs requests that tile the keys; otherwise every row is
    zero, the status is EINVAL and the insert changes nothing."""
    rng = np.random.default_rng(13)
    pair = Pair(10_000, 4)
    toks, off = _rand_prompts(rng, 3, 200, 400)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)
    pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, [0, 1, 2], [1, 2, 3], 1)
    before = pair.gix.dump()
    gapped = to_dev(np.array([0, blk_off[1], blk_off[2], nb - 1], np.int64))  # last block uncovered
    state = pair.gix.probe(d_keys, gapped, nb)
    m = pair.gix.match_probed(state, d_keys, gapped, nb).cpu().numpy()
    assert not m.any()
    pair.gix.insert_probed(state, 3, nb, to_dev(np.array([1, 1, 1], np.int32)), to_dev(np.array([5, 6, 7], np.uint32)), 2)
    n, st = pair.gix.stats()
    assert st == oracle.EINVAL
    after = pair.gix.dump()
    assert all(np.array_equal(a, b) for a, b in zip(before, after))


@pytest.mark.parametrize("B", [16, 8])
def test_reserved_marker_keys(B):
    """Prompts built so that a block's unremapped key is the table's EMPTY (0) or TOMB
    (2^64-1) marker, at block 0, at a 64-block tile edge, mid-prompt and as the last
    block: smetric_hash_blocks and smetric_hash_partition both emit the remapped keys
    (1, 2^64-2) bit for bit with the oracle, and the index stores, matches and refreshes
    those keys like any other (the markers themselves are never written as keys)."""
    from tests.reserved_keys import KEY_EMPTY, KEY_TOMB, prompt_with_reserved
    seed = W.DEFAULT_SEED
    rng = np.random.default_rng(40 + B)
    prompts = [prompt_with_reserved(1, {0: KEY_EMPTY}, seed, B, rng=rng),
               prompt_with_reserved(1, {0: KEY_TOMB}, seed, B, tail=B - 1, rng=rng),
               prompt_with_reserved(130, {0: KEY_TOMB, 63: KEY_EMPTY, 64: KEY_TOMB, 100: KEY_TOMB, 129: KEY_EMPTY},
                                    seed, B, tail=3, rng=rng),
               prompt_with_reserved(70, {69: KEY_TOMB}, seed, B, rng=rng),
               rng.integers(0, W.VOCAB, 40 * B + 9, dtype=np.int32)]
    off = np.zeros(len(prompts) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    toks = np.concatenate(prompts)
    I = 4
    pair = Pair(100_000, I, seed=seed, block=B)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)
    where = {0: [1], 1: [2**64 - 2], 2: [2**64 - 2, 1, 2**64 - 2, 2**64 - 2, 1], 3: [2**64 - 2]}
    pos = {0: [0], 1: [0], 2: [0, 63, 64, 100, 129], 3: [69]}
    for r, ks in where.items():
        got = [int(okeys[blk_off[r] + j]) for j in pos[r]]
        assert got == ks, f"prompt {r}: oracle keys {[hex(k) for k in got]}"
    assert not np.any(okeys == 0) and not np.any(okeys == np.uint64(2**64 - 1))
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    keys, state = pair.gix.hash_partition(to_dev(toks), to_dev(off), d_boff, nb, block_size=B, seed=seed,
                                          status=status)
    assert int(status.item()) == 0
    assert np.array_equal(keys[:nb].cpu().numpy(), okeys), "fused hash + partition keys"
    # enter every prompt on its own instance through the probed path, then route the same
    # prompts again: each sees its whole block sequence on that instance
    pair.gix.probe_lookup(state, keys, d_boff, nb)
    gm = pair.gix.match_probed(state, keys, d_boff, nb).cpu().numpy()
    om = pair.oix.match(okeys, blk_off)
    assert np.array_equal(gm, om) and not gm.any()
    R = len(prompts)
    inst = (np.arange(R) % I).astype(np.int32)
    pair.gix.insert_probed(state, R, nb, to_dev(inst), to_dev(np.arange(R, dtype=np.uint32) + 1), 1)
    assert pair.oix.insert(okeys, blk_off, inst, np.arange(R) + 1, 1) == 0
    pair.compare_index(f"reserved keys B={B}")
    gk, _ = pair.gix.dump()
    assert {1, 2**64 - 2} <= set(int(k) for k in gk)
    nbr = np.diff(blk_off)
    for probed in (False, True):
        b = W.Batch(tokens=toks, tok_off=off, prompt_len=np.diff(off).astype(np.int32),
                    hist_len=np.diff(off).astype(np.int32), turn=np.ones(R, np.int32),
                    session=np.arange(R, dtype=np.uint32) + 1, q=np.zeros(I, np.int64), rr_base=0, epoch=2 + probed)
        pair.step(b, params=dict(W.DEFAULT_PARAMS, block_size=B), what=f"reserved keys again probed={probed}",
                  probed=probed)
        m = pair.oix.match(okeys, blk_off)
        for r in range(R):
            assert m[r][inst[r]] == nbr[r], (r, m[r].tolist())


def test_probe_bound_skips_blocks_and_refreshes_orphans():
    """A prompt whose blocks 16..23 were evicted while the later blocks stayed cached
    (orphans): the lookup's probe bound search (evenly spaced tests, closer than 8 blocks
    apart) lands in the evicted run, so the blocks from there on are not probed; the match
    still equals the oracle's, and the probed insert at the orphans' instance turns the
    unprobed blocks that are entries into refreshes and re-adds the evicted ones -- the
    dump and the entry count equal the oracle's."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(90)
    pair = Pair(10_000, 4)
    toks = rng.integers(0, W.VOCAB, 50 * 16 + 5, dtype=np.int32)
    tok_off = np.array([0, len(toks)], np.int64)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, tok_off)
    # every block on instance 2, blocks 16..23 at epoch 1 (the oldest), the others at 5
    old = np.zeros(nb, bool)
    old[16:24] = True
    for sel, ep in ((~old, 5), (old, 1)):
        k = okeys[sel]
        d = torch.from_numpy(k.view(np.int64)).cuda().view(torch.uint64)
        off = np.array([0, len(k)], np.int64)
        assert pair.insert_both(d, to_dev(off), len(k), k, off, [2], [9], ep) == 0
    pair.gix.evict(4, 25)  # ceil(50 * 4 / 25) = 8 entries
    assert pair.oix.evict(4, 25) == 0
    pair.compare_index("blocks 16..23 evicted")
    assert pair.oix.size == nb - 8
    keys, state = pair.gix.hash_partition(to_dev(toks), to_dev(tok_off), d_boff, nb)
    pair.gix.probe_lookup(state, keys, d_boff, nb)
    probed, searched = S.Index.probe_stats(state, nb)
    assert 16 <= probed < 24 and searched > 0, (probed, searched)
    gm = pair.gix.match_probed(state, keys, d_boff, nb).cpu().numpy()
    om = pair.oix.match(okeys, blk_off)
    assert np.array_equal(gm, om) and gm[0].tolist() == [0, 0, 16, 0]
    pair.gix.insert_probed(state, 1, nb, to_dev(np.array([2], np.int32)), to_dev(np.array([11], np.uint32)), 7)
    assert pair.oix.insert(okeys, blk_off, [2], [11], 7) == 0
    pair.compare_index("orphans refreshed, evicted blocks re-added")
    assert pair.oix.size == nb
    # the same prompt again: every block is held, nothing is skipped
    keys, state = pair.gix.hash_partition(to_dev(toks), to_dev(tok_off), d_boff, nb)
    pair.gix.probe_lookup(state, keys, d_boff, nb)
    probed, _ = S.Index.probe_stats(state, nb)
    assert probed == nb
    gm = pair.gix.match_probed(state, keys, d_boff, nb).cpu().numpy()
    assert gm[0].tolist() == [0, 0, nb, 0]


def test_probe_bound_small_and_empty_requests():
    """Probe bounds over prompts of 0-5 blocks and longer ones, some entered whole, some in
    part, some not at all, with empty requests between them: the match, the route and the
    probed insert equal the oracle's, and the lookup probes no more blocks than exist and
    every block a fully cached prompt has."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(91)
    I = 6
    pair = Pair(50_000, I)
    lens_blk = [0, 1, 2, 3, 0, 5, 1, 40, 0, 2, 17, 64, 65, 0, 3]
    prompts = [rng.integers(0, W.VOCAB, 16 * n + int(rng.integers(0, 16)), dtype=np.int32) for n in lens_blk]
    off = np.zeros(len(prompts) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    toks = np.concatenate(prompts)
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(toks, off)
    # enter a prefix of each prompt: whole (even r), half (r % 3 == 1), none (others)
    R = len(prompts)
    keep = [lens_blk[r] if r % 2 == 0 else (lens_blk[r] // 2 if r % 3 == 1 else 0) for r in range(R)]
    sel = np.concatenate([np.arange(blk_off[r], blk_off[r] + keep[r]) for r in range(R)]).astype(np.int64)
    pk = okeys[sel]
    poff = np.zeros(R + 1, np.int64)
    poff[1:] = np.cumsum(keep)
    d_pk = to_dev(pk)
    inst = (np.arange(R) % I).astype(np.int32)
    assert pair.insert_both(d_pk, to_dev(poff), int(poff[-1]), pk, poff, inst, np.arange(R, dtype=np.uint32), 1) == 0
    keys, state = pair.gix.hash_partition(to_dev(toks), to_dev(off), d_boff, nb)
    pair.gix.probe_lookup(state, keys, d_boff, nb)
    probed, searched = S.Index.probe_stats(state, nb)
    assert probed <= nb and probed >= sum(keep[r] for r in range(R) if r % 2 == 0)
    gm = pair.gix.match_probed(state, keys, d_boff, nb).cpu().numpy()
    om = pair.oix.match(okeys, blk_off)
    assert np.array_equal(gm, om)
    b = W.Batch(tokens=toks, tok_off=off, prompt_len=np.diff(off).astype(np.int32),
                hist_len=np.diff(off).astype(np.int32), turn=np.ones(R, np.int32),
                session=np.arange(R, dtype=np.uint32) + 100, q=rng.integers(0, 10**6, I).astype(np.int64),
                rr_base=3, epoch=2)
    gt, gb = S.route(to_dev(gm), to_dev(b.prompt_len), to_dev(b.hist_len), to_dev(b.turn), to_dev(b.q),
                     W.DEFAULT_PARAMS, b.rr_base)
    ot, ob = oracle.route(om, b.prompt_len, b.hist_len, b.turn, b.q, W.DEFAULT_PARAMS, b.rr_base)
    assert np.array_equal(gt.cpu().numpy(), ot) and np.array_equal(gb.cpu().numpy(), ob)
    pair.gix.insert_probed(state, R, nb, to_dev(np.asarray(ot, np.int32)), to_dev(b.session), b.epoch)
    assert pair.oix.insert(okeys, blk_off, ot, b.session, b.epoch) == 0
    pair.compare_index("small and empty requests")
    say(f"  blocks {nb}, probed {probed}, search probes {searched}")


@pytest.mark.parametrize("I,holders", [(4096, [4095, 2055, 300]), (65536, [65535, 40000, 256])])
def test_refresh_raises_epochs_of_high_instances(I, holders):
    """Refreshes of existing entries on instances whose id has a high byte (the refresh is
    a 32-bit atomic maximum over the value's epoch, kind and instance high byte): plain
    entries and, with I = 4096, bitmap members of a prefix held by more instances than the
    spill threshold; epochs raised on the probed path, then to the largest epoch on the
    self-contained insert, then an older epoch that changes nothing.  Every dump equals
    the oracle's."""
    rng = np.random.default_rng(17 + I)
    pair = Pair(100_000, I)
    pre = rng.integers(0, W.VOCAB, 16 * 32, dtype=np.int32)
    n0 = 48
    others = [i for i in rng.choice(I, n0 + len(holders), replace=False) if i not in holders][: n0 - len(holders)]
    inst = np.array(list(holders) + others, np.int32)
    tails = [rng.integers(0, W.VOCAB, 16 * 6, dtype=np.int32) for _ in range(n0)]
    prompts = [np.concatenate([pre, t]) for t in tails]
    off = np.zeros(n0 + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(np.concatenate(prompts), off)
    assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, inst, np.arange(n0), 5) == 0
    pair.compare_index("entered")
    # follow-ups of the holders' sessions: each sticks to its own instance (q = 0)
    k = len(holders)
    fol = [np.concatenate([prompts[j], rng.integers(0, W.VOCAB, 40, dtype=np.int32)]) for j in range(k)]
    foff = np.zeros(k + 1, np.int64)
    foff[1:] = np.cumsum([len(p) for p in fol])
    for epoch, probed in [(1000, True), ((1 << 22) - 1, False), (7, True)]:
        b = W.Batch(tokens=np.concatenate(fol), tok_off=foff, prompt_len=np.diff(foff).astype(np.int32),
                    hist_len=np.diff(off)[:k].astype(np.int32), turn=np.ones(k, np.int32),
                    session=np.arange(k, dtype=np.uint32), q=np.zeros(I, np.int64), rr_base=0, epoch=epoch)
        ot, ob = pair.step(b, what=f"epoch {epoch}", probed=probed)
        assert list(ot) == list(holders), f"targets {list(ot)}"
