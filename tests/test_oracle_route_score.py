"""Pins for the oracle's comparison scorers of the scoring template (CPU only).

Sec. 4.1 routes a request to the instance minimising a score f of its load and the request's
KV$ hit; the scorers the paper compares against (Sec. 4.1 motivating analysis, Sec. 5
baselines) differ only in f.  Each is pinned by a hand-worked table whose answer a plausible
mistake changes (weights swapped, a hit counted in blocks instead of tokens, the load
normalised by the sum instead of the maximum, a sum instead of a product, >= instead of >
in Preble's half-prompt test), and by the special cases where f reduces to a textbook rule:
round robin when every score ties, join-the-shortest-queue on an empty index, most-cached
with nothing queued, and the weighted sum at lam = 0 (load only) and lam = 1 (hit only).
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle

LOAD, TOKENS, PRODUCT, LINEAR, HIT = (oracle.SCORE_LOAD, oracle.SCORE_TOKENS, oracle.SCORE_PRODUCT,
                                      oracle.SCORE_LINEAR, oracle.SCORE_HIT_FILTER)


def one(kind, c, L, q, load, B=10, lam=(1, 2), rr_base=0):
    t, b = oracle.route_score(kind, np.array([c], np.int32), [L], q, load, B, lam, rr_base)
    return int(t[0]), int(b[0])


def rot_argmin(vals, start):
    """Textbook argmin with the rotation tie-break: the first minimum met walking
    start, start+1, ... (mod I)."""
    I = len(vals)
    order = [(start + k) % I for k in range(I)]
    return min(order, key=lambda i: (vals[i], order.index(i)))


def test_weighted_sum_hand_table():
    """L = 100, B = 10, c = [8, 4, 0] blocks -> hit ratios 0.8, 0.4, 0; batch sizes 10, 5, 0
    -> normalised loads 1, 0.5, 0.
      lam = 1/2: f = 0.6, 0.55, 0.5   -> 2   (normalising by the sum, 15, would give 0)
      lam = 3/4: f = 0.4, 0.575, 0.75 -> 0   (weights swapped would give 2; a hit ratio in
                                              blocks, c/L, would give 2)
      lam = 1/4: f = 0.8, 0.525, 0.25 -> 2"""
    c, load, q = [8, 4, 0], [10, 5, 0], [0, 0, 0]
    assert one(LINEAR, c, 100, q, load, lam=(1, 2)) == (2, 6)
    assert one(LINEAR, c, 100, q, load, lam=(3, 4)) == (0, 6)
    assert one(LINEAR, c, 100, q, load, lam=(1, 4)) == (2, 6)
    # queued work does not enter the weighted sum
    assert one(LINEAR, c, 100, [10**15, 0, 0], load, lam=(3, 4)) == (0, 6)


def test_weighted_sum_exact_tie_takes_rotation_order():
    """lam = 1/2, loads 2, 0, B = 10, L = 100, c = [5, 0]: f0 = 0.5 * 1 + 0.5 * 0.5 = 0.75 and
    f1 = 0 + 0.5 * 1 = 0.5 -> 1.  With c = [10, 0]: f0 = 0.5 = f1, an exact tie, so the
    rotation start decides (a floating-point evaluation could break it either way)."""
    assert one(LINEAR, [5, 0], 100, [0, 0], [2, 0]) == (1, 6)
    assert one(LINEAR, [10, 0], 100, [0, 0], [2, 0], rr_base=0) == (0, 6)
    assert one(LINEAR, [10, 0], 100, [0, 0], [2, 0], rr_base=1) == (1, 6)


def test_tokens_left_hand_table():
    """Dynamo: f = queued tokens + new tokens.  L = 1000, B = 10, c = [80, 0]:
    q = [500, 0] -> f = 700, 1000 -> 0 (a hit in blocks, 1000 - 80, would give 1420 -> 1);
    q = [900, 0] -> f = 1100, 1000 -> 1 (dropping q would give 0)."""
    assert one(TOKENS, [80, 0], 1000, [500, 0], [7, 0]) == (0, 6)
    assert one(TOKENS, [80, 0], 1000, [900, 0], [0, 7]) == (1, 6)


def test_product_hand_table():
    """LMetric: f = (q + L - c) x l.  L = 1000, B = 10, c = [90, 0], q = 0:
    l = [2, 1]  -> 100 * 2 = 200 against 1000 * 1 -> 0;
    l = [20, 1] -> 2000 against 1000 -> 1 (a sum, 120 against 1001, would give 0);
    an idle instance scores 0 and wins whatever its hit."""
    assert one(PRODUCT, [90, 0], 1000, [0, 0], [2, 1]) == (0, 6)
    assert one(PRODUCT, [90, 0], 1000, [0, 0], [20, 1]) == (1, 6)
    assert one(PRODUCT, [90, 0, 0], 1000, [0, 0, 10**12], [20, 1, 0]) == (2, 6)


def test_hit_filter_hand_table():
    """Preble: more than half the prompt cached (strict).  L = 100, B = 10:
    c = [5, 0]: 50 tokens is exactly half -> no filter, the weighted sum decides;
    c = [6, 0]: instance 0 holds 60 > 50 -> it is the only holder and wins at any load;
    c = [9, 6, 0], l = [5, 3, 0]: both 0 and 1 hold more than half -> the less loaded, 1;
    c = [10, 6, 0], l = [4, 3, 0], lam = 3/4: the holders' weighted sums are 0.25 and 0.4875,
    but the filter takes the less loaded holder, 1, not the better score."""
    t, b = one(HIT, [5, 0], 100, [0, 0], [9, 0], lam=(1, 2))
    assert b == 6 and (t, b) == one(LINEAR, [5, 0], 100, [0, 0], [9, 0], lam=(1, 2))
    assert one(HIT, [6, 0], 100, [0, 0], [10**6, 0]) == (0, 7)
    assert one(HIT, [9, 6, 0], 100, [0, 0, 0], [5, 3, 0]) == (1, 7)
    assert one(LINEAR, [10, 6, 0], 100, [0, 0, 0], [4, 3, 0], lam=(3, 4)) == (0, 6)
    assert one(HIT, [10, 6, 0], 100, [0, 0, 0], [4, 3, 0], lam=(3, 4)) == (1, 7)


def test_special_cases_reduce_to_textbook_rules():
    rng = np.random.default_rng(8101)
    for trial in range(300):
        I = int(rng.integers(1, 9))
        B = int(rng.choice([2, 4, 16, 64]))
        L = int(rng.integers(1, 4000))
        c = rng.integers(0, L // B + 1, size=I)
        q = rng.integers(0, 50, size=I)
        load = rng.integers(0, 6, size=I)
        rr = int(rng.integers(0, 2**64 - 1, dtype=np.uint64))
        start = rr % I
        # every score equal -> round robin from the rotation start
        assert one(LOAD, c, L, q, [3] * I, B, rr_base=rr)[0] == start
        # load only
        assert one(LOAD, c, L, q, load, B, rr_base=rr)[0] == rot_argmin(list(load), start)
        # weighted sum at lam = 0 is load only, at lam = 1 the most-cached instance
        assert one(LINEAR, c, L, q, load, B, (0, 5), rr)[0] == rot_argmin(list(load), start)
        assert one(LINEAR, c, L, q, load, B, (5, 5), rr)[0] == rot_argmin(list(-c), start)
        # fewest tokens on an empty index is join-the-shortest-queue on queued tokens;
        # with nothing queued it is the most-cached instance
        assert one(TOKENS, [0] * I, L, q, load, B, rr_base=rr)[0] == rot_argmin(list(q), start)
        assert one(TOKENS, c, L, [0] * I, load, B, rr_base=rr)[0] == rot_argmin(list(-c), start)
        # the product with equal positive loads is the fewest-tokens rule
        assert (one(PRODUCT, c, L, q, [4] * I, B, rr_base=rr)[0] ==
                one(TOKENS, c, L, q, load, B, rr_base=rr)[0])
        # Preble without a holder of more than half the prompt is the weighted sum
        lam = (int(rng.integers(0, 8)), 7)
        if not np.any(2 * B * c > L):
            assert one(HIT, c, L, q, load, B, lam, rr) == one(LINEAR, c, L, q, load, B, lam, rr)


def test_weighted_sum_against_fractions():
    """The weighted sum evaluated term by term in exact rationals (fractions.Fraction),
    including an idle cluster (max load 0) and empty prompts."""
    rng = np.random.default_rng(8102)
    for trial in range(300):
        I = int(rng.integers(1, 7))
        B = 4
        L = int(rng.integers(0, 200))
        c = rng.integers(0, L // B + 1, size=I)
        load = rng.integers(0, 4, size=I) * int(rng.integers(0, 2))
        lam = Fraction(int(rng.integers(0, 9)), 8)
        lmax = int(load.max())
        lhat = [Fraction(int(x), lmax) if lmax else Fraction(0) for x in load]
        chat = [Fraction(B * int(x), L) if L else Fraction(0) for x in c]
        f = [(1 - lam) * lhat[i] + lam * (1 - chat[i]) for i in range(I)]
        rr = int(rng.integers(0, 1000))
        assert one(LINEAR, c, L, [0] * I, load, B, (lam.numerator, lam.denominator), rr)[0] == \
            rot_argmin(f, rr % I)


def test_domain_and_errors():
    q, load = [0, 0], [1, 1]
    assert one(TOKENS, [0, 11], 100, q, load) == (-1, 255)      # c above L / B
    assert one(TOKENS, [0, 0], -1, q, load) == (-1, 255)
    assert one(TOKENS, [0, 0], (1 << 24) + 1, q, load) == (-1, 255)
    assert one(LOAD, [0, 0], 100, [0, 1 << 62], load) == (-1, 255)
    assert one(PRODUCT, [0, 0], 100, q, [1, -1]) == (-1, 255)
    assert one(LINEAR, [10, 0], 100, q, [2**31 - 1, 0], lam=(2**31 - 1, 2**31 - 1)) == (0, 6)
    t, b = oracle.route_score(LOAD, np.zeros((0, 3), np.int32), [], [0] * 3, [0] * 3, 16)
    assert t.size == 0 and b.size == 0
    for bad in [dict(kind=5), dict(kind=-1), dict(B=3), dict(B=258), dict(kind=LINEAR, lam=(2, 1)),
                dict(kind=HIT, lam=(0, 0)), dict(kind=LINEAR, lam=(-1, 2))]:
        a = dict(dict(kind=LOAD, B=16, lam=(1, 2)), **bad)
        with pytest.raises(ValueError):
            oracle.route_score(a["kind"], np.zeros((1, 2), np.int32), [10], q, load, a["B"], a["lam"])
    # lam is not checked for the scorers that do not use it
    assert oracle.route_score(TOKENS, np.zeros((1, 2), np.int32), [10], q, load, 16, (0, 0))[1][0] == 6
