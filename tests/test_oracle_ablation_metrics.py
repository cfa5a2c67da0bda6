"""Pins for the oracle's Sec. 5.4 load-aware filter and the Sec. 4.1 load-imbalance metric
(CPU only).

Load-aware filter ("overloading migration" of the ablation): the basic session-centric
rule sticks a cached follow-up to its previous instance; the filter makes it leave when
that instance's load exceeds the cluster mean by a margin.  Pins: the decision table; an
infinite margin is the basic rule; an even load never triggers it (load = mean is not
above it); the exact threshold load > mean (1 + m); leaving and first turns balance exactly
as the Sec. 4.2 rule's balance (pinned separately).

Imbalance: the load of an instance in a window is its average number of running requests,
the imbalance the maximum over the mean.  Pins: hand-computed overlaps; a perfectly even
assignment gives 1; everything on one instance gives I; conservation (the window sums add
up to the total running time inside the windows).
"""
import numpy as np

import oracle

P = dict(c_lin=100_000, c_att=3, slo_b=1_000_000_000, slo_a=62_500,
         slack_num=1, slack_den=1, hit_num=1, hit_den=2, block_size=16)


def la1(c, L, hist, turn, q, load, margin, rr=0):
    t, b = oracle.route_loadaware(np.array([c], np.int32), [L], [hist], [turn], q, load, margin, P, rr)
    return int(t[0]), int(b[0])


def test_decision_table():
    L, hist, c = 1200, 960, [60, 0, 0]
    q = [0, 0, 10]
    assert la1(c, L, hist, 0, q, [0, 0, 0], (1, 2)) == (0, 0)           # first turn: balance
    assert la1([30, 0, 0], L, 961, 1, q, [0, 0, 0], (1, 2)) == (0, 1)   # evicted: balance
    assert la1(c, L, hist, 2, q, [100, 100, 100], (1, 2)) == (0, 2)     # even load: stick
    # prev's load 300 vs mean 400/3: above mean x 1.5 = 200 -> leave to the balance target
    t, b = la1(c, L, hist, 2, [10**10, 0, 10], [300, 50, 50], (1, 2))
    assert (t, b) == (1, 4)


def test_exact_threshold_and_infinite_margin():
    L, hist, c = 1200, 960, [60, 0, 0, 0]
    # loads [x, 100, 100, 100], margin 1/2: leave iff x * 4 * 2 > (x + 300) * 3  <=>  5x > 900
    assert la1(c, L, hist, 1, [0] * 4, [180, 100, 100, 100], (1, 2))[1] == 2   # 900 = 900: stays
    assert la1(c, L, hist, 1, [0] * 4, [181, 100, 100, 100], (1, 2))[1] == 4
    # margin 0: leave iff strictly above the mean
    assert la1(c, L, hist, 1, [0] * 4, [100, 100, 100, 100], (0, 1))[1] == 2
    assert la1(c, L, hist, 1, [0] * 4, [101, 100, 100, 100], (0, 1))[1] == 4
    # infinite margin (den 0): the basic session-centric rule never leaves
    assert la1(c, L, hist, 1, [0] * 4, [10**15, 0, 0, 0], (1, 0))[1] == 2


def test_balance_targets_are_the_main_rule():
    rng = np.random.default_rng(4)
    R, I = 400, 23
    L = rng.integers(0, 3000, R).astype(np.int32)
    m = np.minimum(rng.integers(0, 200, (R, I)), (L // 16)[:, None]).astype(np.int32)
    hist = rng.integers(0, 3000, R).astype(np.int32)
    turn = rng.integers(0, 3, R).astype(np.int32)
    q = rng.integers(0, 100, I).astype(np.int64) * 20_000_000
    load = rng.integers(0, 1000, I).astype(np.int64)
    t, b = oracle.route_loadaware(m, L, hist, turn, q, load, (1, 4), P, 99)
    tb, bb = oracle.route(m, L, hist, np.zeros(R, np.int32), q, P, 99)
    moved = np.isin(b, [0, 1, 4])
    assert np.array_equal(t[moved], tb[moved])
    stay = b == 2
    assert np.array_equal(t[stay], m[stay].argmax(axis=1))
    assert set(b.tolist()) <= {0, 1, 2, 4}


def test_imbalance_hand_computed():
    # window 10: request 0 on instance 0 runs [0, 25) -> windows 0, 1 full, window 2 half
    # request 1 on instance 1 runs [5, 15) -> 5 in window 0, 5 in window 1
    s, mx, bad = oracle.imbalance([0, 1], [0, 5], [25, 15], 2, 10, 3)
    assert s.tolist() == [15, 15, 5] and mx.tolist() == [10, 10, 5] and bad == 0


def test_imbalance_even_and_concentrated():
    I, R, W = 8, 800, 10
    rng = np.random.default_rng(2)
    t0 = rng.integers(0, 900, R)
    t1 = t0 + rng.integers(1, 300, R)
    # every request on one instance: max = sum, so max / mean = I
    s, mx, _ = oracle.imbalance(np.zeros(R, np.int32), t0, t1, I, 100, W)
    assert np.array_equal(mx, s)
    # the same request pattern copied on every instance: max / mean = 1
    inst = np.repeat(np.arange(I, dtype=np.int32), R)
    s, mx, _ = oracle.imbalance(inst, np.tile(t0, I), np.tile(t1, I), I, 100, W)
    assert np.array_equal(mx * I, s)
    # conservation: the window sums add up to the running time inside [0, W x window)
    s, _, _ = oracle.imbalance(rng.integers(0, I, R), t0, t1, I, 100, W)
    assert s.sum() == int(np.minimum(t1, W * 100).sum() - np.minimum(t0, W * 100).sum())


def test_imbalance_skips_bad_requests():
    s, mx, bad = oracle.imbalance([0, 5, -1, 1], [0, 0, 0, 10], [10, 10, 10, 5], 2, 10, 1)
    assert bad == 3 and s.tolist() == [10] and mx.tolist() == [10]
