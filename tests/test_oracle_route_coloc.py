"""Pins for the oracle's route under PD colocation (CPU only).

App. B's pseudocode differs from Sec. 4.2's in three places, and each is pinned against a
value the text fixes or a rule it reduces to:
* a TPOT candidate filter: the new request's prefill (Eq. (1) with n = L - hit) stalls an
  instance's live decodes and must fit their smallest slack; an instance without live
  decodes always passes (all() over nothing), and when no instance passes the filter is
  dropped;
* LMetric's multiplicative score (estimate_load x the instance's request count, Sec. 4.1
  and App. B) picks the balance target;
* no last-resort clause: with SLACK = 0 every follow-up migrates (Sec. 5.5's statement),
  and SLACK = inf ignores the TTFT check.
Reductions: with every instance free of decodes and equal request counts the balance
target is the Sec. 4.2 rule's (already pinned); with zero request counts every score is 0
and the target is the rotation start (rr_base + r) mod I.
"""
import numpy as np

import oracle

P = dict(c_lin=100_000, c_att=3, slo_b=1_000_000_000, slo_a=62_500,
         slack_num=1, slack_den=1, hit_num=1, hit_den=2, block_size=16)
FREE = oracle.NO_DECODE


def cost(L, hit_tokens, c_lin=P["c_lin"], c_att=P["c_att"]):
    """Eq. (1) in ns of prefill time (exact, as a float of an exact half-integer)."""
    n = L - hit_tokens
    return c_lin * n + c_att * n * (L - n / 2)


def coloc1(c, L, hist, turn, q, slack, n_run, rr_base=0, **over):
    p = dict(P, **over)
    t, b = oracle.route_coloc(np.array([c], np.int32), [L], [hist], [turn], q, slack, n_run, p, rr_base)
    return int(t[0]), int(b[0])


def test_decision_table():
    L, hist = 1200, 960
    c = [60, 0, 0]  # instance 0 holds the previous prompt
    free3, one3 = [FREE] * 3, [1, 1, 1]
    assert coloc1(c, L, hist, 0, [0, 0, 0], free3, one3) == (0, 0)          # first turn: balance
    assert coloc1([30, 0, 0], L, 961, 1, [0, 0, 0], free3, one3) == (0, 1)  # evicted: balance
    assert coloc1(c, L, hist, 3, [10**9, 0, 0], free3, one3) == (0, 2)      # stick
    # prev misses its TTFT deadline -> migrate to the lowest score
    assert coloc1(c, L, hist, 3, [5 * 10**9, 0, 10], free3, one3) == (1, 4)
    # nobody meets TTFT: no last resort under colocation, still migrate
    assert coloc1(c, L, hist, 3, [5 * 10**9] * 3, free3, one3)[1] == 4
    # prev meets TTFT but fails the TPOT filter while instance 2 passes -> migrate (5)
    stall0 = cost(L, 960)
    assert coloc1(c, L, hist, 3, [0, 0, 0], [int(stall0) - 1, 0, FREE], one3) == (2, 5)


def test_tpot_filter_boundary_is_the_prefill_stall():
    """meets_tpot: stall = prefill_cost(req, c[i]) <= smallest decode slack.  L = 1,201 with
    c = 60 blocks leaves n = 241 new tokens; the stall 1e5 * 241 + 3 * 241 * (1201 - 120.5) is a
    half-integer, so the slack floor(stall) fails and floor(stall) + 1 passes."""
    L, c = 1201, [60, 0]
    stall = cost(L, 960)
    assert stall != int(stall)
    lo = int(stall)
    # instance 1 holds nothing and has no decodes; make it the worse balance choice
    q = [0, 10**12]
    assert coloc1(c, L, 960, 2, q, [lo + 1, FREE], [1, 1]) == (0, 2)  # passes: stick
    assert coloc1(c, L, 960, 2, q, [lo, FREE], [1, 1]) == (1, 5)      # fails: the filter moves it
    # the stall is the request's own prefill: the instance's queue does not count
    q = [10**6, 10**12]
    assert coloc1(c, L, 960, 2, q, [lo + 1, FREE], [1, 1]) == (0, 2)


def test_no_instance_passes_drops_the_filter():
    L, c = 1200, [60, 0, 0]
    # every instance has a decode with negative slack: nothing passes, so cand = all and prev sticks
    assert coloc1(c, L, 960, 1, [0, 0, 0], [-1, -1, -1], [1, 1, 1]) == (0, 2)
    # first turn: balance over all instances by score
    assert coloc1(c, L, 960, 0, [0, 0, 0], [-1, -1, -1], [1, 1, 1]) == (0, 0)


def test_multiplicative_score_of_lmetric():
    """est(0) = 10 units with 5 requests (score 50) loses to est(1) = 20 units with 2 requests
    (score 40), although instance 0 has the smaller estimated load (c_lin = 0, c_att = 0, so
    est = q)."""
    kw = dict(c_lin=0, c_att=0)
    assert coloc1([0, 0], 64, 0, 0, [10, 20], [FREE, FREE], [5, 2], **kw) == (1, 0)
    assert coloc1([0, 0], 64, 0, 0, [10, 20], [FREE, FREE], [3, 2], **kw) == (0, 0)   # 30 < 40
    assert coloc1([0, 0], 64, 0, 0, [10, 20], [FREE, FREE], [4, 2], **kw) == (0, 0)   # tie 40 = 40: rotation start 0
    assert coloc1([0, 0], 64, 0, 0, [10, 20], [FREE, FREE], [4, 2], rr_base=1, **kw) == (1, 0)
    # an idle instance (no requests) scores 0 whatever its queue
    assert coloc1([0, 0, 0], 64, 0, 0, [10, 5, 10**9], [FREE] * 3, [1, 1, 0], **kw) == (2, 0)


def test_slack_zero_every_followup_migrates():
    """Sec. 5.5: SLACK = 0 disables stickiness -- every follow-up with a positive estimated
    load migrates (under colocation there is no last-resort stick)."""
    rng = np.random.default_rng(11)
    R, I = 200, 16
    m = rng.integers(0, 80, (R, I)).astype(np.int32)
    L = np.full(R, 1280, np.int32)
    hist = np.zeros(R, np.int32)  # always cached
    turn = np.ones(R, np.int32)
    q = rng.integers(1, 10**9, I).astype(np.int64)
    t, b = oracle.route_coloc(m, L, hist, turn, q, np.full(I, FREE), np.ones(I, np.int32),
                              dict(P, slack_num=0, slack_den=1))
    assert set(b.tolist()) == {4}


def test_slack_inf_ignores_ttft():
    """SLACK = inf: the TTFT check always passes, so a cached follow-up sticks unless the
    TPOT filter excludes its instance."""
    L, c = 1200, [60, 0]
    huge = [10**17, 0]
    assert coloc1(c, L, 960, 1, huge, [FREE, FREE], [1, 1], slack_num=1, slack_den=0) == (0, 2)
    assert coloc1(c, L, 960, 1, huge, [FREE, FREE], [1, 1]) == (1, 4)


def test_reduces_to_the_main_rule_balance_without_decodes():
    """No live decodes and equal request counts: argmin of est x k is argmin of est, so
    first-turn targets equal the Sec. 4.2 rule's balance targets (pinned separately)."""
    rng = np.random.default_rng(5)
    R, I = 300, 37
    m = rng.integers(0, 60, (R, I)).astype(np.int32)
    L = np.full(R, 1024, np.int32)
    hist = np.zeros(R, np.int32)
    turn = np.zeros(R, np.int32)
    q = (rng.integers(0, 4, I) * 10**6).astype(np.int64)  # many exact ties
    t_main, b_main = oracle.route(m, L, hist, turn, q, P, 17)
    for k in (1, 7):
        t, b = oracle.route_coloc(m, L, hist, turn, q, np.full(I, FREE), np.full(I, k, np.int32), P, 17)
        assert np.array_equal(t, t_main) and set(b.tolist()) == {0}


def test_idle_fleet_is_round_robin():
    """Every instance without requests: all scores are 0 and the target is the rotation start."""
    R, I = 50, 9
    m = np.zeros((R, I), np.int32)
    t, _ = oracle.route_coloc(m, np.full(R, 512, np.int32), np.zeros(R, np.int32), np.zeros(R, np.int32),
                              np.arange(I, dtype=np.int64) * 10**6, np.full(I, FREE), np.zeros(I, np.int32), P, 4)
    assert np.array_equal(t, (4 + np.arange(R)) % I)


def test_out_of_domain_inputs():
    L, c = 1200, [60, 0]
    assert coloc1(c, L, 960, 1, [0, 0], [FREE, FREE], [1, -1]) == (-1, 255)   # negative request count
    assert coloc1([80, 0], L, 960, 1, [0, 0], [FREE, FREE], [1, 1]) == (-1, 255)  # c > L / B
