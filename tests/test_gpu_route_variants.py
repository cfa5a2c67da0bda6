"""GPU route variants (through the C ABI) vs the CPU oracle, bit for bit: the rule under
PD colocation (App. B).  Random batches cover every branch, both sides of the TPOT
filter (instances without decodes, slacks around the prefill stall, slacks nobody meets),
idle instances (score 0), instance counts that are not multiples of the 64-lane wave,
128-bit extremes and out-of-domain inputs; one case routes the matched rows of a real
session workload."""
import numpy as np
import pytest

import oracle
from paper_2607_08565_amd import workload as W
from tests.parity import Pair, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _coloc_inputs(rng, R, I, L_hi=4000):
    L = rng.integers(0, L_hi, R).astype(np.int32)
    m = rng.integers(0, L_hi // 16 + 1, (R, I)).astype(np.int32)
    m = np.minimum(m, (L // 16)[:, None]).astype(np.int32)
    hist = rng.integers(0, L_hi, R).astype(np.int32)
    turn = rng.integers(0, 3, R).astype(np.int32)
    q = (rng.integers(0, 200, I) * W.Q_UNIT_NS).astype(np.int64)
    # slacks: a third without decodes, a third around typical stalls, the rest anywhere
    kind = rng.integers(0, 3, I)
    slack = np.where(kind == 0, oracle.NO_DECODE,
                     np.where(kind == 1, rng.integers(0, 4 * 10**8, I), rng.integers(-10**9, 10**10, I))).astype(np.int64)
    n_run = rng.integers(0, 40, I).astype(np.int32)
    return m, L, hist, turn, q, slack, n_run


def _both(S, m, L, hist, turn, q, slack, n_run, p, rr):
    gt, gb = S.route_coloc(to_dev(m), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q), to_dev(slack),
                           to_dev(n_run), p, rr)
    ot, ob = oracle.route_coloc(m, L, hist, turn, q, slack, n_run, p, rr)
    gt, gb = gt.cpu().numpy(), gb.cpu().numpy()
    bad = np.nonzero((gt != ot) | (gb != ob))[0]
    assert len(bad) == 0, f"{len(bad)} decisions differ, first {bad[:5]}: gpu {gt[bad[:3]]}/{gb[bad[:3]]} oracle {ot[bad[:3]]}/{ob[bad[:3]]}"
    return ot, ob


@pytest.mark.parametrize("I", [1, 3, 64, 65, 1000, 5000])
def test_coloc_random_parity(I):
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(100 + I)
    R = 1500 if I <= 1000 else 300
    m, L, hist, turn, q, slack, n_run = _coloc_inputs(rng, R, I)
    seen = set()
    for over in ({}, dict(slack_num=0, slack_den=1), dict(slack_num=1, slack_den=0), dict(c_att=0, c_lin=1),
                 dict(slack_num=3, slack_den=2, hit_num=0, hit_den=5)):
        p = dict(W.DEFAULT_PARAMS, **over)
        for rr in (0, 987654321):
            _, ob = _both(S, m, L, hist, turn, q, slack, n_run, p, rr)
            seen |= set(ob.tolist())
    # every slack below any stall: the filter is dropped
    _both(S, m, L, hist, turn, q, np.full(I, -1, np.int64), n_run, W.DEFAULT_PARAMS, 5)
    # an idle fleet: every score is 0
    _both(S, m, L, hist, turn, q, slack, np.zeros(I, np.int32), W.DEFAULT_PARAMS, 5)
    say(f"  I={I}: branches seen {sorted(seen)}")
    assert {0, 1, 2, 4} <= seen
    if I in (64, 1000, 5000):
        assert 5 in seen


def test_coloc_extremes_and_out_of_domain():
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(7)
    R, I = 200, 70
    L = np.full(R, 1 << 24, np.int32)
    L[:50] = rng.integers(0, 1 << 24, 50)
    m = rng.integers(0, (1 << 24) // 256 + 1, (R, I)).astype(np.int32)
    m = np.minimum(m, (L // 256)[:, None]).astype(np.int32)
    hist = rng.integers(0, 1 << 24, R).astype(np.int32)
    turn = rng.integers(0, 2, R).astype(np.int32)
    q = rng.integers((1 << 62) - 10**6, 1 << 62, I).astype(np.int64)
    slack = rng.integers(-(1 << 62), 1 << 62, I).astype(np.int64)
    slack[::5] = np.iinfo(np.int64).max
    n_run = rng.integers(0, 2**31 - 1, I).astype(np.int32)
    big = dict(W.DEFAULT_PARAMS, c_lin=1 << 32, c_att=1 << 32, slo_b=1 << 32, slo_a=1 << 32, block_size=256,
               slack_num=2**31 - 1, slack_den=1)
    _both(S, m, L, hist, turn, q, slack, n_run, big, 2**64 - 1)
    # out of domain: c above L / B, negative turn, and a negative request count (all requests)
    m2 = m.copy()
    m2[3, 1] = L[3] // 256 + 1
    t2 = turn.copy()
    t2[4] = -1
    _, ob = _both(S, m2, L, hist, t2, q, slack, n_run, big, 0)
    assert ob[3] == 255 and ob[4] == 255
    n_bad = n_run.copy()
    n_bad[10] = -1
    _, ob = _both(S, m, L, hist, turn, q, slack, n_bad, big, 0)
    assert set(ob.tolist()) == {255}


def test_coloc_on_matched_rows_of_a_session_workload():
    """Route the real c rows of a scaled mid-fleet workload (closed loop) under colocation."""
    from paper_2607_08565_amd import smetric as S
    wl = W.config1(n_sess=256, n_turns=3)
    pair = Pair(4_000_000, wl.n_inst)
    rng = np.random.default_rng(3)
    prev = None
    for t in range(3):
        b = wl.batch(t, prev)
        d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(b.tokens, b.tok_off)
        gm = pair.gix.match(d_keys, d_boff, nb)
        om = pair.oix.match(okeys, blk_off)
        assert np.array_equal(gm.cpu().numpy(), om)
        slack = rng.integers(0, 2 * 10**9, wl.n_inst).astype(np.int64)
        slack[rng.random(wl.n_inst) < 0.3] = oracle.NO_DECODE
        n_run = rng.integers(0, 30, wl.n_inst).astype(np.int32)
        ot, ob = _both(S, om, b.prompt_len, b.hist_len, b.turn, b.q, slack, n_run, W.DEFAULT_PARAMS, b.rr_base)
        say(f"  batch {t}: branches {np.bincount(ob, minlength=6).tolist()}")
        pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, ot, b.session, b.epoch)
        prev = ot


# ---------------------------------------------------------------------------------
# Online load update (requests routed one at a time)
# ---------------------------------------------------------------------------------
def _seq_both(S, m, L, hist, turn, q, p, rr):
    gt, gb, gq = S.route_seq(to_dev(m), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q), p, rr)
    ot, ob, oq = oracle.route_seq(m, L, hist, turn, q, p, rr)
    gt, gb, gq = gt.cpu().numpy(), gb.cpu().numpy(), gq.cpu().numpy()
    bad = np.nonzero((gt != ot) | (gb != ob))[0]
    assert len(bad) == 0, f"{len(bad)} decisions differ, first {bad[:5]}: gpu {gt[bad[:3]]}/{gb[bad[:3]]} oracle {ot[bad[:3]]}/{ob[bad[:3]]}"
    assert np.array_equal(gq, oq), "final loads differ"
    return ot, ob


@pytest.mark.parametrize("I", [1, 3, 64, 65, 1000, 1024, 1025, 4096])
def test_seq_random_parity(I):
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(200 + I)
    R = 3000 if I <= 1025 else 800
    m, L, hist, turn, q, _, _ = _coloc_inputs(rng, R, I)
    seen = set()
    for over in ({}, dict(slack_num=0, slack_den=1), dict(slack_num=1, slack_den=0), dict(c_att=0, c_lin=1),
                 dict(slack_num=3, slack_den=2, hit_num=0, hit_den=5)):
        p = dict(W.DEFAULT_PARAMS, **over)
        for rr in (0, 987654321):
            _, ob = _seq_both(S, m, L, hist, turn, q, p, rr)
            seen |= set(ob.tolist())
    say(f"  I={I}: branches seen {sorted(seen)}")
    assert {0, 1, 2, 3} <= seen
    if I > 1:
        assert 4 in seen


@pytest.mark.parametrize("I", [2, 4, 37])
def test_seq_blocks_of_cached_follow_ups(I):
    """Cached follow-ups only, on few instances: most requests of every 64-request block
    share a prev, and the queues cross deadlines inside blocks, so the block-wise decisions
    (loads accumulated over earlier requests with the same prev) meet the sequential rule's
    sticks, last resorts and migrations; a sprinkle of first turns and out-of-domain rows."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(300 + I)
    R = 5000
    L = rng.integers(1024, 8192, R).astype(np.int32)
    prev = rng.integers(0, I, R)
    m = (rng.integers(0, 30, (R, I)) * (L // 16)[:, None] // 100).astype(np.int32)
    m[np.arange(R), prev] = (L // 16) * rng.integers(60, 100, R) // 100
    hist = (L * 6 // 10).astype(np.int32)  # c[prev] * 16 > hist / 2: cached
    turn = np.ones(R, np.int32)
    turn[rng.random(R) < 0.01] = 0
    m[rng.random(R) < 0.005, 0] = 1 << 20  # out of domain (c > L / B)
    q = rng.integers(0, 40, I).astype(np.int64) * W.Q_UNIT_NS
    seen = set()
    # the last two make per-request costs exceed 2^32 ns (words with bit 31 set cross lanes)
    for over in ({}, dict(slack_num=1, slack_den=2), dict(slack_num=4, slack_den=1), dict(c_lin=20_000),
                 dict(c_lin=4_000_000, slo_b=2**32), dict(c_lin=4_000_000, c_att=3_000, slo_b=2**32, slo_a=2**32)):
        p = dict(W.DEFAULT_PARAMS, **over)
        _, ob = _seq_both(S, m, L, hist, turn, q, p, 12345)
        seen |= set(ob.tolist())
    say(f"  I={I}: branches seen {sorted(seen)}")
    assert {0, 2, 3, 255} <= seen


def test_seq_extremes_invalid_and_limits():
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(8)
    R, I = 300, 70
    L = np.full(R, 1 << 24, np.int32)
    L[:50] = rng.integers(0, 1 << 24, 50)
    m = np.minimum(rng.integers(0, (1 << 24) // 256 + 1, (R, I)), (L // 256)[:, None]).astype(np.int32)
    hist = rng.integers(0, 1 << 24, R).astype(np.int32)
    turn = rng.integers(0, 2, R).astype(np.int32)
    q = rng.integers((1 << 62) - 10**6, 1 << 62, I).astype(np.int64)
    big = dict(W.DEFAULT_PARAMS, c_lin=1 << 32, c_att=1 << 32, slo_b=1 << 32, slo_a=1 << 32, block_size=256,
               slack_num=2**31 - 1, slack_den=1)
    _seq_both(S, m, L, hist, turn, q, big, 2**64 - 1)  # loads far beyond 2^64 (saturated q_out)
    m2, t2 = m.copy(), turn.copy()
    m2[3, 1] = L[3] // 256 + 1
    t2[4] = -1
    _, ob = _seq_both(S, m2, L, hist, t2, q, big, 0)
    assert ob[3] == 255 and ob[4] == 255
    qb = q.copy()
    qb[0] = -1
    _, ob = _seq_both(S, m, L, hist, turn, qb, big, 0)
    assert set(ob.tolist()) == {255}
    with pytest.raises(S.SmetricError):
        S.route_seq(to_dev(np.zeros((2, 4097), np.int32)), to_dev(np.zeros(2, np.int32)),
                    to_dev(np.zeros(2, np.int32)), to_dev(np.zeros(2, np.int32)), to_dev(np.zeros(4097, np.int64)),
                    W.DEFAULT_PARAMS)
    # an empty batch leaves the loads as they were
    gt, gb, gq = S.route_seq(to_dev(np.zeros((0, 5), np.int32)), to_dev(np.zeros(0, np.int32)),
                             to_dev(np.zeros(0, np.int32)), to_dev(np.zeros(0, np.int32)),
                             to_dev(np.arange(5, dtype=np.int64)), W.DEFAULT_PARAMS)
    assert gq.cpu().numpy().tolist() == list(range(5))


@pytest.mark.parametrize("I", [64, 1000])
def test_seq_loads_crossing_2_pow_49(I):
    """Loads that start just under 2^49 ns and grow past it within the batch: scans move
    from the range where every score 2q + est2 stays below 2^51 (computed in double
    precision) to the 128-bit one mid-batch; first turns only (a scan per request), then the
    random mix of turns."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(500 + I)
    R = 2000
    m, L, hist, turn, _, _, _ = _coloc_inputs(rng, R, I)
    q = rng.integers((1 << 49) - 3 * (1 << 38), (1 << 49) - (1 << 38), I).astype(np.int64)
    # first turns on small hits (costly), with the costs scaled to cross within the batch
    for over in (dict(c_lin=(1 << 24) * (I // 64)), dict(c_lin=(1 << 23) * (I // 64), c_att=(1 << 12) * (I // 64))):
        _, ob = _seq_both(S, m // 4, L, hist, np.zeros_like(turn), q, dict(W.DEFAULT_PARAMS, **over), 77)
        assert set(ob.tolist()) <= {0, 255}
    for over in (dict(c_lin=1 << 28), dict(c_lin=1 << 27, c_att=1 << 16)):
        _seq_both(S, m, L, hist, turn, q, dict(W.DEFAULT_PARAMS, **over), 78)


def test_seq_on_matched_rows_of_a_session_workload():
    """Online routing of the real c rows of a scaled long-context workload, closed loop."""
    from paper_2607_08565_amd import smetric as S
    wl = W.config2(n_sess=128, n_turns=3, l0=4096, app=(512, 2048), prefix_len=2048)
    pair = Pair(4_000_000, wl.n_inst)
    prev = None
    for t in range(3):
        b = wl.batch(t, prev)
        d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(b.tokens, b.tok_off)
        om = pair.oix.match(okeys, blk_off)
        assert np.array_equal(pair.gix.match(d_keys, d_boff, nb).cpu().numpy(), om)
        ot, ob = _seq_both(S, om, b.prompt_len, b.hist_len, b.turn, b.q, W.DEFAULT_PARAMS, b.rr_base)
        bt, _ = oracle.route(om, b.prompt_len, b.hist_len, b.turn, b.q, W.DEFAULT_PARAMS, b.rr_base)
        say(f"  batch {t}: branches {np.bincount(ob, minlength=5).tolist()}, "
            f"{int((bt != ot).sum())} of {len(ot)} targets differ from the batch-snapshot rule")
        pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, ot, b.session, b.epoch)
        prev = ot


# ---------------------------------------------------------------------------------
# Colocation rule, requests routed one at a time (App. B)
# ---------------------------------------------------------------------------------
def _seqc_both(S, m, L, hist, turn, q, slack, n_run, p, rr):
    gt, gb, gq, gn = S.route_seq_coloc(to_dev(m), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q), to_dev(slack),
                                       to_dev(n_run), p, rr)
    ot, ob, oq, on = oracle.route_seq_coloc(m, L, hist, turn, q, slack, n_run, p, rr)
    gt, gb, gq, gn = gt.cpu().numpy(), gb.cpu().numpy(), gq.cpu().numpy(), gn.cpu().numpy()
    bad = np.nonzero((gt != ot) | (gb != ob))[0]
    assert len(bad) == 0, f"{len(bad)} decisions differ, first {bad[:5]}: gpu {gt[bad[:3]]}/{gb[bad[:3]]} oracle {ot[bad[:3]]}/{ob[bad[:3]]}"
    assert np.array_equal(gq, oq), "final loads differ"
    assert np.array_equal(gn, on), "final request counts differ"
    return ot, ob


@pytest.mark.parametrize("I", [1, 3, 64, 65, 1000, 1024, 1025, 4096])
def test_seqc_random_parity(I):
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(400 + I)
    R = 3000 if I <= 1025 else 800
    m, L, hist, turn, q, slack, n_run = _coloc_inputs(rng, R, I)
    seen = set()
    for over in ({}, dict(slack_num=0, slack_den=1), dict(slack_num=1, slack_den=0), dict(c_att=0, c_lin=1),
                 dict(slack_num=3, slack_den=2, hit_num=0, hit_den=5)):
        p = dict(W.DEFAULT_PARAMS, **over)
        for rr in (0, 987654321):
            _, ob = _seqc_both(S, m, L, hist, turn, q, slack, n_run, p, rr)
            seen |= set(ob.tolist())
    _seqc_both(S, m, L, hist, turn, q, np.full(I, -1, np.int64), n_run, W.DEFAULT_PARAMS, 5)  # nobody passes
    _seqc_both(S, m, L, hist, turn, q, slack, np.zeros(I, np.int32), W.DEFAULT_PARAMS, 5)  # an idle fleet
    say(f"  I={I}: branches seen {sorted(seen)}")
    assert {0, 1, 2, 4} <= seen
    if I >= 64:
        assert 5 in seen


@pytest.mark.parametrize("R", [1, 2, 31, 32, 33, 63, 64, 65, 97])
def test_seqc_batch_sizes_around_block_edges(R):
    """Batches of 1 to 97 requests: the last block partial or full, one to four blocks, on
    a fleet larger than a candidate list and on one smaller."""
    from paper_2607_08565_amd import smetric as S
    for I in (7, 200):
        rng = np.random.default_rng(1000 * R + I)
        m, L, hist, turn, q, slack, n_run = _coloc_inputs(rng, R, I)
        _seqc_both(S, m, L, hist, turn, q, slack, n_run, W.DEFAULT_PARAMS, 17 * R)


@pytest.mark.parametrize("I", [2, 4, 37, 150])
def test_seqc_blocks_of_cached_follow_ups(I):
    """Cached follow-ups whose prev is a candidate, on few instances: most requests of
    every 64-request step share a prev and the queues cross deadlines inside steps, so the
    step-wise sticks meet the sequential rule's migrations; some prevs fail the TPOT filter,
    a sprinkle of first turns and out-of-domain rows."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(500 + I)
    R = 5000
    L = rng.integers(1024, 8192, R).astype(np.int32)
    prev = rng.integers(0, I, R)
    m = (rng.integers(0, 30, (R, I)) * (L // 16)[:, None] // 100).astype(np.int32)
    m[np.arange(R), prev] = (L // 16) * rng.integers(60, 100, R) // 100
    hist = (L * 6 // 10).astype(np.int32)
    turn = np.ones(R, np.int32)
    turn[rng.random(R) < 0.01] = 0
    m[rng.random(R) < 0.005, 0] = 1 << 20  # out of domain (c > L / B)
    q = rng.integers(0, 40, I).astype(np.int64) * W.Q_UNIT_NS
    slack = np.full(I, oracle.NO_DECODE, np.int64)
    slack[0] = 10**8  # instance 0 fails the filter for the longer stalls
    n_run = rng.integers(0, 20, I).astype(np.int32)
    seen = set()
    for over in ({}, dict(slack_num=1, slack_den=2), dict(slack_num=4, slack_den=1), dict(c_lin=20_000),
                 dict(c_lin=4_000_000, slo_b=2**32), dict(c_lin=4_000_000, c_att=3_000, slo_b=2**32, slo_a=2**32)):
        p = dict(W.DEFAULT_PARAMS, **over)
        _, ob = _seqc_both(S, m, L, hist, turn, q, slack, n_run, p, 12345)
        seen |= set(ob.tolist())
    say(f"  I={I}: branches seen {sorted(seen)}")
    assert {0, 2, 4, 255} <= seen


@pytest.mark.parametrize("I", [129, 300, 1000, 2049])
def test_seqc_identical_requests_exhaust_candidate_lists(I):
    """Identical requests rank the instances alike, so the earlier requests of a block and of
    the block before take the best listed candidates of the later ones: the regime where
    the minimum over a request's list (its best candidates on the state before the previous
    block, rescored) must still equal the minimum over all instances."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(900 + I)
    R = 4000
    m = np.zeros((R, I), np.int32)
    L = np.full(R, 8192, np.int32)
    z = np.zeros(R, np.int32)
    for q, n_run in ((np.zeros(I, np.int64), np.zeros(I, np.int32)),
                     (rng.integers(0, 10**9, I).astype(np.int64), rng.integers(0, 5, I).astype(np.int32))):
        slack = np.full(I, oracle.NO_DECODE, np.int64)
        ot, ob = _seqc_both(S, m, L, z, z, q, slack, n_run, W.DEFAULT_PARAMS, 11)
        assert set(ob.tolist()) == {0}
        assert len(np.unique(ot[:I])) > I // 2  # the first ones spread over the fleet


def test_seqc_scores_past_128_bits_and_limits():
    """140,000 maximal prefills on two instances with nearly 2^31 requests each: the LMetric
    products pass 2^127, where only the exact comparison keeps both sides equal; then the
    state-domain, size and overflow limits and the empty batch."""
    from paper_2607_08565_amd import smetric as S
    R, I = 140_000, 2
    big = dict(W.DEFAULT_PARAMS, c_lin=1 << 32, c_att=1 << 32, block_size=256)
    m = np.zeros((R, I), np.int32)
    L = np.full(R, 1 << 24, np.int32)
    z = np.zeros(R, np.int32)
    q = np.zeros(I, np.int64)
    slack = np.full(I, oracle.NO_DECODE, np.int64)
    n_run = np.array([2**31 - 1, 2**31 - 3], np.int32)
    ot, _ = _seqc_both(S, m, L, z, z, q, slack, n_run, big, 0)
    cost2 = 2 * (1 << 32) * (1 << 24) + (1 << 32) * (1 << 48)
    assert int(np.bincount(ot, minlength=2).max()) * cost2 * 2**31 > 2**127  # past 128 bits
    n_bad = n_run.copy()
    n_bad[1] = -1
    _, ob = _seqc_both(S, m[:100], L[:100], z[:100], z[:100], q, slack, n_bad, big, 0)
    assert set(ob.tolist()) == {255}
    with pytest.raises(S.SmetricError):  # more instances than the LDS holds
        S.route_seq_coloc(to_dev(np.zeros((2, 4097), np.int32)), to_dev(np.zeros(2, np.int32)),
                          to_dev(np.zeros(2, np.int32)), to_dev(np.zeros(2, np.int32)),
                          to_dev(np.zeros(4097, np.int64)), to_dev(np.zeros(4097, np.int64)),
                          to_dev(np.zeros(4097, np.int32)), W.DEFAULT_PARAMS)
    with pytest.raises(S.SmetricError):  # loads that could overflow the deadline check
        huge = dict(big, slack_num=1, slack_den=2**31 - 1)
        S.route_seq_coloc(to_dev(m), to_dev(L), to_dev(z), to_dev(z), to_dev(q), to_dev(slack), to_dev(n_run), huge)
    gt, gb, gq, gn = S.route_seq_coloc(to_dev(np.zeros((0, 5), np.int32)), to_dev(np.zeros(0, np.int32)),
                                       to_dev(np.zeros(0, np.int32)), to_dev(np.zeros(0, np.int32)),
                                       to_dev(np.arange(5, dtype=np.int64)), to_dev(np.zeros(5, np.int64)),
                                       to_dev(np.arange(5, dtype=np.int32)), W.DEFAULT_PARAMS)
    assert gq.cpu().numpy().tolist() == list(range(5)) and gn.cpu().numpy().tolist() == list(range(5))


def test_seqc_on_matched_rows_of_a_session_workload():
    """The colocated rule one request at a time on the real c rows of a scaled mid-fleet
    workload (closed loop), against the batch-snapshot rule for reference."""
    from paper_2607_08565_amd import smetric as S
    wl = W.config1(n_sess=256, n_turns=3)
    pair = Pair(4_000_000, wl.n_inst)
    rng = np.random.default_rng(13)
    prev = None
    for t in range(3):
        b = wl.batch(t, prev)
        d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(b.tokens, b.tok_off)
        om = pair.oix.match(okeys, blk_off)
        assert np.array_equal(pair.gix.match(d_keys, d_boff, nb).cpu().numpy(), om)
        slack = rng.integers(0, 2 * 10**9, wl.n_inst).astype(np.int64)
        slack[rng.random(wl.n_inst) < 0.3] = oracle.NO_DECODE
        n_run = rng.integers(0, 30, wl.n_inst).astype(np.int32)
        ot, ob = _seqc_both(S, om, b.prompt_len, b.hist_len, b.turn, b.q, slack, n_run, W.DEFAULT_PARAMS, b.rr_base)
        bt, _ = oracle.route_coloc(om, b.prompt_len, b.hist_len, b.turn, b.q, slack, n_run, W.DEFAULT_PARAMS, b.rr_base)
        say(f"  batch {t}: branches {np.bincount(ob, minlength=6).tolist()}, "
            f"{int((bt != ot).sum())} of {len(ot)} targets differ from the batch-snapshot rule")
        pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, ot, b.session, b.epoch)
        prev = ot


# ---------------------------------------------------------------------------------
# Sec. 5.4 ablation: load-aware filter; Sec. 4.1 load-imbalance metric
# ---------------------------------------------------------------------------------
@pytest.mark.parametrize("I", [1, 3, 64, 65, 1000, 5000])
def test_loadaware_random_parity(I):
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(300 + I)
    R = 1500 if I <= 1000 else 300
    m, L, hist, turn, q, _, _ = _coloc_inputs(rng, R, I)
    load = rng.integers(0, 10**9, I).astype(np.int64)
    seen = set()
    for margin in ((1, 2), (0, 1), (1, 0), (7, 3)):
        for rr in (0, 12345):
            gt, gb = S.route_loadaware(to_dev(m), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q), to_dev(load),
                                       margin, W.DEFAULT_PARAMS, rr)
            ot, ob = oracle.route_loadaware(m, L, hist, turn, q, load, margin, W.DEFAULT_PARAMS, rr)
            assert np.array_equal(gt.cpu().numpy(), ot) and np.array_equal(gb.cpu().numpy(), ob), (margin, rr)
            seen |= set(ob.tolist())
    assert {0, 1, 2} <= seen
    if I > 1:
        assert 4 in seen
    # a load outside its range: every request out of domain
    bad = load.copy()
    bad[0] = -1
    gt, gb = S.route_loadaware(to_dev(m), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q), to_dev(bad), (1, 2),
                               W.DEFAULT_PARAMS)
    assert set(gb.cpu().numpy().tolist()) == {255}


@pytest.mark.parametrize("I,W_", [(1, 1), (7, 5), (64, 100), (1000, 37)])
def test_imbalance_parity(I, W_):
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(I * 31 + W_)
    R = 20000
    inst = rng.integers(-2, I + 2, R).astype(np.int32)  # some out of range
    t0 = rng.integers(-500, 120 * W_, R).astype(np.int64)
    t1 = t0 + rng.integers(-5, 400, R)  # some negative durations, some zero
    window = 100
    gs, gm, gb = S.imbalance(to_dev(inst), to_dev(t0), to_dev(t1), I, window, W_)
    os_, om, ob = oracle.imbalance(inst, t0, t1, I, window, W_)
    assert np.array_equal(gs.cpu().numpy(), os_) and np.array_equal(gm.cpu().numpy(), om)
    assert int(gb.item()) == ob
