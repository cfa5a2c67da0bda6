"""Pins for the oracle's route with the online load update (CPU only).

Sec. 4.2 (a) routes one request at a time against q, the prefill already queued at each
instance; a routed request's prefill (Eq. (1), reusing its hit on the target) joins the
target's queue before the next request is routed.  Pins:
* a hand-worked water-filling case (costs C, queues 0 and 1.5 C: targets 0, 0, 1);
* with one request, or when every later request's decision is independent of load
  (SLACK = inf and cached follow-ups), the batch rule's decisions;
* every decision equals the batch rule applied to that single request with the queue
  rebuilt from the earlier decisions (the batch rule is pinned separately), and the final
  queue is the initial one plus the routed costs;
* identical first-turn requests on an equally loaded fleet spread round-robin;
* out-of-domain requests add no load.
"""
import numpy as np

import oracle

P = dict(c_lin=100_000, c_att=3, slo_b=1_000_000_000, slo_a=62_500,
         slack_num=1, slack_den=1, hit_num=1, hit_den=2, block_size=16)


def cost2(L, c, p=P):
    """2 x Eq. (1) with n = L - B c, as a Python integer."""
    n = L - p["block_size"] * c
    return 2 * p["c_lin"] * n + p["c_att"] * n * (2 * L - n)


def test_water_filling_by_hand():
    p = dict(P, c_lin=1000, c_att=0, slo_b=10**9, slo_a=0)
    C = 16_000  # 16 new tokens x 1,000 ns
    t, b, q = oracle.route_seq(np.zeros((3, 2), np.int32), [16] * 3, [0] * 3, [0] * 3, [0, 3 * C // 2], p, 0)
    assert t.tolist() == [0, 0, 1] and b.tolist() == [0, 0, 0]
    assert q.tolist() == [2 * C, 3 * C // 2 + C]
    # the batch rule sends all three to the least loaded instance of the snapshot
    tb, _ = oracle.route(np.zeros((3, 2), np.int32), [16] * 3, [0] * 3, [0] * 3, [0, 3 * C // 2], p, 0)
    assert tb.tolist() == [0, 0, 0]


def test_single_request_equals_batch_rule():
    rng = np.random.default_rng(1)
    for _ in range(50):
        I = int(rng.integers(1, 40))
        L = int(rng.integers(0, 3000))
        c = rng.integers(0, L // 16 + 1, (1, I)).astype(np.int32)
        q = rng.integers(0, 100, I).astype(np.int64) * 20_000_000
        args = (c, [L], [int(rng.integers(0, 3000))], [int(rng.integers(0, 3))], q)
        t, b, _ = oracle.route_seq(*args, P, 7)
        tb, bb = oracle.route(*args, P, 7)
        assert (t[0], b[0]) == (tb[0], bb[0])


def test_load_independent_decisions_match_batch():
    """SLACK = inf and every request a cached follow-up: each sticks whatever the loads."""
    rng = np.random.default_rng(2)
    R, I = 300, 20
    L = np.full(R, 1600, np.int32)
    m = rng.integers(0, 50, (R, I)).astype(np.int32)
    m[np.arange(R), rng.integers(0, I, R)] = 100  # a clear holder per request
    hist = np.full(R, 1600, np.int32)  # 100 blocks * 16 = 1600 > 1600 / 2: cached
    turn = np.ones(R, np.int32)
    q = rng.integers(0, 100, I).astype(np.int64) * 20_000_000
    p = dict(P, slack_num=1, slack_den=0)
    t, b, _ = oracle.route_seq(m, L, hist, turn, q, p, 0)
    tb, bb = oracle.route(m, L, hist, turn, q, p, 0)
    assert np.array_equal(t, tb) and set(b.tolist()) == {2}


def test_each_decision_is_the_batch_rule_on_the_rebuilt_queue():
    rng = np.random.default_rng(3)
    for trial in range(4):
        R, I = 120, int(rng.integers(2, 30))
        L = (rng.integers(0, 2000, R) * 2).astype(np.int32)  # even L: every cost is a whole ns
        m = np.minimum(rng.integers(0, 250, (R, I)), (L // 16)[:, None]).astype(np.int32)
        hist = rng.integers(0, 4000, R).astype(np.int32)
        turn = rng.integers(0, 3, R).astype(np.int32)
        q = rng.integers(0, 60, I).astype(np.int64) * 20_000_000
        rr = int(rng.integers(0, 2**40))
        t, b, q_after = oracle.route_seq(m, L, hist, turn, q, P, rr)
        q2 = [2 * int(x) for x in q]  # doubled, exact
        for r in range(R):
            # the batch rule for request r alone, with the rebuilt queue
            assert all(v % 2 == 0 for v in q2)
            qq = np.array([v // 2 for v in q2], np.int64)
            tb, bb = oracle.route(m[r:r + 1], L[r:r + 1], hist[r:r + 1], turn[r:r + 1], qq, P, rr + r)
            assert (t[r], b[r]) == (tb[0], bb[0]), (trial, r)
            q2[t[r]] += cost2(int(L[r]), int(m[r, t[r]]))
        assert q_after.tolist() == [v // 2 for v in q2]


def test_identical_first_turns_spread_round_robin():
    R, I = 40, 7
    m = np.zeros((R, I), np.int32)
    t, b, q = oracle.route_seq(m, np.full(R, 800, np.int32), np.zeros(R, np.int32), np.zeros(R, np.int32),
                               np.zeros(I, np.int64), P, 3)
    assert np.array_equal(t, (3 + np.arange(R)) % I)
    per = cost2(800, 0) // 2
    counts = np.bincount(t, minlength=I)
    assert q.tolist() == [int(k) * per for k in counts]


def test_out_of_domain_requests_add_no_load():
    m = np.zeros((3, 2), np.int32)
    m[1, 0] = 1000  # c > L / B
    t, b, q = oracle.route_seq(m, [160, 160, 160], [0, 0, 0], [0, 0, 0], [0, 0], P, 0)
    assert b.tolist() == [0, 255, 0] and t.tolist() == [0, -1, 1]
    assert q.tolist() == [cost2(160, 0) // 2] * 2
