"""Pins for the oracle's route step (CPU only).

Sec. 4.2's pseudocode, parts (a) routing, (b) SLO checks and (c) load model, with
Eq. (1) as the prefill cost.  The paper prints no numeric routing example, so the cases
are built by hand from the rule and checked against values it fixes:
* the 3-token prompt with 2 cached tokens computes 1 token (Sec. 2);
* raising reuse from 70 % to 80 % cuts the tokens still to compute by a third (Sec. 4.1);
* Eq. (1) closed forms: cost(0, L) = 0, cost(L, L) = c_lin L + c_att L^2 / 2;
* the TTFT SLO b + a L with b = 1 s, a = 62.5 ms per 1K tokens: 2.0 s at 16,000 tokens (Sec. 5.2);
* special cases: an empty index reduces to join-the-shortest-queue (Sec. 4.1), c_att = 0
  to fewest-tokens-left, SLACK = inf to plain session stickiness (Sec. 5.4/5.5), and
  SLACK = 0 to the listing's last-resort stick (its "none meets" clause).
"""
import numpy as np
import pytest

import oracle

P = dict(c_lin=100_000, c_att=3, slo_b=1_000_000_000, slo_a=62_500,
         slack_num=1, slack_den=1, hit_num=1, hit_den=2, block_size=16)
STICK_BRANCHES = {2, 3}


def route1(c, L, hist, turn, q, rr_base=0, **over):
    p = dict(P, **over)
    t, b = oracle.route(np.array([c], np.int32), [L], [hist], [turn], q, p, rr_base)
    return int(t[0]), int(b[0])


def test_decision_table_five_branches():
    # instance 0 holds the session's previous prompt (c = 60 blocks = 960 tokens of 1,200)
    L, hist = 1200, 960
    c = [60, 0, 0]
    # 1. first turn -> balance by estimated load (instance 0 has the smallest load)
    assert route1(c, L, hist, 0, [0, 0, 0]) == (0, 0)
    # 2. follow-up whose hit is not above HIT_RATIO * est_hit -> evicted, balance
    assert route1([30, 0, 0], L, 961, 1, [0, 0, 0]) == (0, 1)  # 480 * 2 > 961 fails
    assert route1([31, 0, 0], L, 961, 1, [0, 0, 0])[1] == 2    # 496 * 2 > 961 holds
    # 3. cached and prev meets the deadline -> stick
    assert route1(c, L, hist, 3, [10**9, 0, 0]) == (0, 2)
    # 4. cached, prev misses, some other instance meets -> migrate to the least loaded
    assert route1(c, L, hist, 3, [5 * 10**9, 0, 10]) == (1, 4)
    # 5. cached, nobody meets -> last-resort stick
    assert route1(c, L, hist, 3, [5 * 10**9, 5 * 10**9, 5 * 10**9]) == (0, 3)


def test_three_token_prompt_with_two_hits_costs_one_token():
    """Sec. 2: 3 tokens, 2 cached -> 1 to compute.  With B = 2, c = 1 block = 2 tokens,
    n = 1 and 2*cost = 2*c_lin + c_att*1*(2*3 - 1).  Instance 1 (nothing cached, n = 3,
    2*cost = 6*c_lin + 9*c_att) ties instance 0 exactly when q1 = q0 - 2*c_lin - 2*c_att."""
    cl, ca, q0 = 1000, 7, 10**6
    tie = q0 - 2 * cl - 2 * ca
    kw = dict(block_size=2, c_lin=cl, c_att=ca)
    assert route1([1, 0], 3, 0, 0, [q0, tie], rr_base=0, **kw)[0] == 0      # tie -> rotation start 0
    assert route1([1, 0], 3, 0, 0, [q0, tie], rr_base=1, **kw)[0] == 1      # tie -> rotation start 1
    assert route1([1, 0], 3, 0, 0, [q0, tie - 1], rr_base=0, **kw)[0] == 1  # strictly cheaper
    assert route1([1, 0], 3, 0, 0, [q0, tie + 1], rr_base=1, **kw)[0] == 0


def test_reuse_70_to_80_percent_cuts_compute_by_a_third():
    """With c_att = 0 the cost is linear in new tokens; L = 1,600 tokens, 70 % cached leaves
    480 tokens, 80 % leaves 320 = 2/3 of 480.  Instances tie when their queues differ by
    c_lin * 160, the third that was cut."""
    L = 1600
    c70, c80 = 70, 80  # blocks of 16
    cl = 1000
    base = 10**8
    q = [base, base + cl * (480 - 320)]  # instance 0 has 70 %, instance 1 has 80 %
    assert route1([c70, c80], L, 0, 0, q, rr_base=0, c_att=0, c_lin=cl)[0] == 0
    assert route1([c70, c80], L, 0, 0, q, rr_base=1, c_att=0, c_lin=cl)[0] == 1
    q[1] += 1
    assert route1([c70, c80], L, 0, 0, q, rr_base=1, c_att=0, c_lin=cl)[0] == 0


def test_eq1_closed_forms_and_slo_at_16000_tokens():
    """L = 16,000: ttft_slo = 1 s + 16 * 62.5 ms = 2.0 s.  Instance 0 holds all 1,000 blocks
    (cost(0, L) = 0), so it meets iff q0 <= 2.0 s.  Instance 1 holds nothing:
    cost(L, L) = 1e5 * 16,000 + 3 * 16,000^2 / 2 = 1.984 s, so it meets iff q1 <= 16 ms."""
    L, c = 16000, [1000, 0]
    two_s = 2_000_000_000
    assert route1(c, L, L, 1, [two_s, 0]) == (0, 2)
    assert route1(c, L, L, 1, [two_s + 1, 0]) == (1, 4)
    assert route1(c, L, L, 1, [two_s + 1, 16_000_000]) == (1, 4)
    assert route1(c, L, L, 1, [two_s + 1, 16_000_001]) == (0, 3)
    # SLACK scales the deadline: SLACK = 1/2 -> 1.0 s for instance 0
    assert route1(c, L, L, 1, [10**9, 10**12], slack_num=1, slack_den=2) == (0, 2)
    assert route1(c, L, L, 1, [10**9 + 1, 10**12], slack_num=1, slack_den=2) == (0, 3)


def test_empty_index_is_join_shortest_queue_with_rotation():
    I, R = 5, 12
    c = np.zeros((R, I), np.int32)
    L = np.full(R, 1000, np.int32)
    q = np.zeros(I, np.int64)
    t, b = oracle.route(c, L, np.zeros(R, np.int32), np.zeros(R, np.int32), q, P, rr_base=3)
    assert t.tolist() == [(3 + r) % I for r in range(R)]
    assert set(b.tolist()) == {0}
    # follow-ups with nothing cached are "evicted" and also balanced
    t, b = oracle.route(c, L, np.full(R, 500, np.int32), np.ones(R, np.int32), q, P, rr_base=3)
    assert t.tolist() == [(3 + r) % I for r in range(R)] and set(b.tolist()) == {1}
    q = np.array([5, 3, 9, 3, 4], np.int64) * 10**6
    t, _ = oracle.route(c[:3], L[:3], np.zeros(3, np.int32), np.zeros(3, np.int32), q, P, rr_base=0)
    # least loaded are 1 and 3; rotation start r picks the first of them at or after r
    assert t.tolist() == [1, 1, 3]


def test_fewest_tokens_left_when_attention_cost_is_zero():
    """c_att = 0, c_lin = 1 ns: estimated load = queued ns + tokens left to prefill."""
    L = 800
    c = [10, 40, 0]          # tokens left: 640, 160, 800
    q = [0, 600, 0]          # totals: 640, 760, 800
    assert route1(c, L, 0, 0, q, c_att=0, c_lin=1)[0] == 0
    q = [0, 400, 0]          # totals: 640, 560, 800
    assert route1(c, L, 0, 0, q, c_att=0, c_lin=1)[0] == 1


def test_slack_infinity_ignores_slo_and_zero_makes_last_resort():
    c, L, hist = [60, 0], 1200, 960
    heavy = [10**15, 0]
    assert route1(c, L, hist, 2, heavy, slack_num=0, slack_den=0) == (0, 2)  # SLACK = inf: stick
    # SLACK = 0: no instance with positive load meets, so the listing's last resort sticks
    assert route1(c, L, hist, 2, [5, 7], slack_num=0, slack_den=1) == (0, 3)


def test_argmax_prefers_lowest_instance_on_ties():
    assert route1([0, 50, 50], 1000, 100, 1, [0, 0, 0]) == (1, 2)
    assert route1([7, 7, 7], 1000, 100, 1, [0, 0, 0]) == (0, 2)


def test_invalid_requests_and_parameters():
    t, b = oracle.route(np.array([[5, 0], [0, 0], [0, 0], [0, 0]], np.int32), [50, -1, 10, 10], [0, 0, -3, 0],
                        [1, 0, 1, -1], [0, 0], P)
    assert t.tolist() == [-1, -1, -1, -1] and b.tolist() == [255] * 4  # c > L/B, L < 0, hist < 0, turn < 0
    t, b = oracle.route(np.zeros((1, 2), np.int32), [10], [0], [0], [0, 1 << 62], P)
    assert b.tolist() == [255]
    for bad in (dict(hit_num=2, hit_den=2), dict(hit_den=0), dict(block_size=15), dict(c_att=-1),
                dict(c_lin=(1 << 32) + 1), dict(slack_num=-1)):
        with pytest.raises(ValueError):
            oracle.route(np.zeros((1, 2), np.int32), [10], [0], [0], [0, 0], dict(P, **bad))


def test_extreme_values_do_not_overflow():
    L = 1 << 24
    big = dict(c_lin=1 << 32, c_att=1 << 32, slo_b=1 << 32, slo_a=1 << 32,
               slack_num=2**31 - 1, slack_den=2**31 - 1, hit_num=2**31 - 2, hit_den=2**31 - 1)
    t, b = oracle.route(np.array([[L // 16, 0]], np.int32), [L], [L], [1], [(1 << 62) - 1, 0], dict(P, **big))
    # instance 0: est = q0 (huge) vs bound ~ 2^56 -> misses; instance 1: cost ~ 2^79 -> misses -> last resort
    assert (t.tolist(), b.tolist()) == ([0], [3])
