"""Pins for the oracle's colocation rule with requests taken one at a time (CPU only).

App. B's router handles one request at a time (req = receive()); its state per instance is
the queued prefill q, the number of requests num_requests, and the slack of the live
decodes.  After a request is forwarded its prefill joins the target's queue and it is one
more request there; its own decode is not live yet, so the slacks stay.  Pins:
* a hand-worked case where the online rule and the batch rule part ways (an idle instance
  scores 0 under LMetric's product until it takes a request);
* with one request, the batch colocation rule (pinned separately);
* when no decision depends on the state (SLACK = inf, cached follow-ups whose prev passes
  the TPOT filter), the batch rule's decisions;
* every decision equals the batch rule applied to that single request on the queue and
  request counts rebuilt from the earlier decisions, and the final state is the initial
  one plus the routed costs and requests;
* out-of-domain requests leave the state unchanged.
"""
import numpy as np

import oracle
from paper_2607_08565_amd.workload import NO_DECODE

P = dict(c_lin=100_000, c_att=3, slo_b=1_000_000_000, slo_a=62_500,
         slack_num=1, slack_den=1, hit_num=1, hit_den=2, block_size=16)


def cost2(L, c, p=P):
    """2 x Eq. (1) with n = L - B c, as a Python integer."""
    n = L - p["block_size"] * c
    return 2 * p["c_lin"] * n + p["c_att"] * n * (2 * L - n)


def test_idle_instance_by_hand():
    p = dict(P, c_lin=1000, c_att=0, slo_b=10**9, slo_a=0)
    C = 16_000  # a 16-token first turn at 1,000 ns per token
    m = np.zeros((3, 2), np.int32)
    args = (m, [16] * 3, [0] * 3, [0] * 3, [0, 0], [NO_DECODE, NO_DECODE], [0, 1])
    t, b, q, n = oracle.route_seq_coloc(*args, p, 0)
    # r0: scores (0 + C) x 0 = 0 and (0 + C) x 1 -> 0; then q0 = C, n0 = 1
    # r1: (C + C) x 1 = 2C and (0 + C) x 1 = C -> 1; then q1 = C, n1 = 2
    # r2: (C + C) x 1 = 2C and (C + C) x 2 = 4C -> 0
    assert t.tolist() == [0, 1, 0] and b.tolist() == [0, 0, 0]
    assert q.tolist() == [2 * C, C] and n.tolist() == [2, 2]
    tb, _ = oracle.route_coloc(*args, p, 0)
    assert tb.tolist() == [0, 0, 0]  # the batch snapshot keeps scoring instance 0 at 0


def _random_case(rng, R, I):
    L = (rng.integers(0, 2000, R) * 2).astype(np.int32)  # even L: every cost is a whole ns
    m = np.minimum(rng.integers(0, 250, (R, I)), (L // 16)[:, None]).astype(np.int32)
    hist = rng.integers(0, 4000, R).astype(np.int32)
    turn = rng.integers(0, 3, R).astype(np.int32)
    q = rng.integers(0, 60, I).astype(np.int64) * 20_000_000
    slack = np.where(rng.random(I) < 0.3, NO_DECODE, rng.integers(0, 3_000_000_000, I)).astype(np.int64)
    n_run = rng.poisson(4, I).astype(np.int32)
    return m, L, hist, turn, q, slack, n_run


def test_single_request_equals_batch_rule():
    rng = np.random.default_rng(1)
    for _ in range(60):
        I = int(rng.integers(1, 40))
        args = _random_case(rng, 1, I)
        t, b, _, _ = oracle.route_seq_coloc(*args, P, 9)
        tb, bb = oracle.route_coloc(*args, P, 9)
        assert (t[0], b[0]) == (tb[0], bb[0])


def test_state_independent_decisions_match_batch():
    rng = np.random.default_rng(2)
    R, I = 300, 20
    L = np.full(R, 1600, np.int32)
    m = rng.integers(0, 50, (R, I)).astype(np.int32)
    m[np.arange(R), rng.integers(0, I, R)] = 100  # a clear holder per request
    hist = np.full(R, 1600, np.int32)  # 100 blocks * 16 = 1600 > 1600 / 2: cached
    turn = np.ones(R, np.int32)
    q = rng.integers(0, 100, I).astype(np.int64) * 20_000_000
    slack = np.full(I, NO_DECODE, np.int64)  # no live decodes: every instance passes the TPOT filter
    n_run = rng.poisson(4, I).astype(np.int32)
    p = dict(P, slack_num=1, slack_den=0)
    t, b, _, n_after = oracle.route_seq_coloc(m, L, hist, turn, q, slack, n_run, p, 0)
    tb, bb = oracle.route_coloc(m, L, hist, turn, q, slack, n_run, p, 0)
    assert np.array_equal(t, tb) and set(b.tolist()) == {2}
    assert np.array_equal(n_after - n_run, np.bincount(t, minlength=I))


def test_each_decision_is_the_batch_rule_on_the_rebuilt_state():
    rng = np.random.default_rng(3)
    for trial in range(4):
        R, I = 120, int(rng.integers(2, 30))
        m, L, hist, turn, q, slack, n_run = _random_case(rng, R, I)
        rr = int(rng.integers(0, 2**40))
        t, b, q_after, n_after = oracle.route_seq_coloc(m, L, hist, turn, q, slack, n_run, P, rr)
        qs = [int(x) for x in q]  # whole ns: every cost of an even L is
        ns = [int(x) for x in n_run]
        for r in range(R):
            tb, bb = oracle.route_coloc(m[r: r + 1], L[r: r + 1], hist[r: r + 1], turn[r: r + 1],
                                        np.array(qs, np.int64), slack, np.array(ns, np.int32), P, rr + r)
            assert (t[r], b[r]) == (tb[0], bb[0]), f"trial {trial} request {r}"
            qs[t[r]] += cost2(int(L[r]), int(m[r, t[r]])) // 2
            ns[t[r]] += 1
        assert q_after.tolist() == qs and n_after.tolist() == ns
        assert set(b.tolist()) <= {0, 1, 2, 4, 5}


def test_out_of_domain_requests_change_nothing():
    rng = np.random.default_rng(4)
    I = 6
    m, L, hist, turn, q, slack, n_run = _random_case(rng, 3, I)
    L = L.copy()
    L[1] = -5  # request 1 out of domain
    t, b, q_after, n_after = oracle.route_seq_coloc(m, L, hist, turn, q, slack, n_run, P, 0)
    assert b[1] == 255 and t[1] == -1 and b[0] != 255 and b[2] != 255
    # the final state is the initial one plus requests 0 and 2 only
    qs, ns = [int(x) for x in q], [int(x) for x in n_run]
    for r in (0, 2):
        qs[t[r]] += cost2(int(L[r]), int(m[r, t[r]])) // 2
        ns[t[r]] += 1
    assert q_after.tolist() == qs and n_after.tolist() == ns


def test_score_comparison_is_exact_past_128_bits():
    """The LMetric product of a running state can pass 2^127 (loads and counts both grow);
    the oracle compares it in 192 bits: checked against Python integers."""
    rng = np.random.default_rng(5)
    for _ in range(2000):
        a, b = (int(v) for v in rng.integers(0, 2**63, 2, dtype=np.uint64))
        a = (a << 64) | int(rng.integers(0, 2**63, dtype=np.uint64))
        b = (b << 64) | int(rng.integers(0, 2**63, dtype=np.uint64))
        x, y = (int(v) for v in rng.integers(0, 2**63, 2, dtype=np.uint64))
        if rng.random() < 0.3:
            b, y = a, x + int(rng.integers(-1, 2))  # near ties
            y = max(y, 0)
        assert oracle.test_prod_less(a, x, b, y) == (a * x < b * y)


def test_batches_whose_loads_could_overflow_are_refused():
    """Both one-at-a-time rules accept a batch only if its largest reachable load, times
    SLACK's denominator, stays below 2^126 (checked here with Python integers at the edge)."""
    import pytest
    big = dict(P, c_lin=2**32, c_att=2**32, slack_num=1, slack_den=2**31 - 1)
    cmax = 2 * 2**32 * 2**24 + 2**32 * 2**48  # the largest doubled cost of a request in domain

    def fits(R):
        return (2**63 + (R + 1) * cmax) * (2**31 - 1) < 2**126

    R_ok = (2**126 // (2**31 - 1) - 2**63) // cmax - 1
    while not fits(R_ok):
        R_ok -= 1
    while fits(R_ok + 1):
        R_ok += 1
    for R, ok in ((R_ok, True), (R_ok + 1, False)):
        m = np.zeros((R, 1), np.int32)
        z = np.zeros(R, np.int32)
        args = (m, z, z, z, np.zeros(1, np.int64))
        if ok:
            oracle.route_seq(*args, big, 0)
            oracle.route_seq_coloc(*args, np.full(1, NO_DECODE, np.int64), np.zeros(1, np.int32), big, 0)
        else:
            with pytest.raises(ValueError):
                oracle.route_seq(*args, big, 0)
            with pytest.raises(ValueError):
                oracle.route_seq_coloc(*args, np.full(1, NO_DECODE, np.int64), np.zeros(1, np.int32), big, 0)
