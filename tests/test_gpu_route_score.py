"""GPU comparison scorers of the scoring template (smetric_route_score, through the C ABI)
vs the CPU oracle, bit for bit, for all five scorers: random batches with many exact ties
(small load and queue ranges, so the rotation tie-break decides often), hit-filter holders
on both sides of the strict half-prompt test, idle clusters and empty prompts (the weighted
sum's normalisers at 0), instance counts around the 64-lane wave and up to the 65,536
limit, 128-bit extremes, every out-of-domain input, host errors, and the matched rows of a
real session workload."""
import numpy as np
import pytest

import oracle
from paper_2607_08565_amd import workload as W
from tests.parity import Pair, say, to_dev

pytestmark = pytest.mark.gpu

KINDS = (oracle.SCORE_LOAD, oracle.SCORE_TOKENS, oracle.SCORE_PRODUCT, oracle.SCORE_LINEAR,
         oracle.SCORE_HIT_FILTER)


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _both(S, kind, m, L, q, load, B, lam, rr):
    gt, gb = S.route_score(kind, to_dev(m), to_dev(L), to_dev(q), to_dev(load), B, lam, rr)
    ot, ob = oracle.route_score(kind, m, L, q, load, B, lam, rr)
    gt, gb = gt.cpu().numpy(), gb.cpu().numpy()
    bad = np.nonzero((gt != ot) | (gb != ob))[0]
    assert len(bad) == 0, (f"kind {kind}: {len(bad)} decisions differ, first {bad[:5]}: "
                           f"gpu {gt[bad[:3]]}/{gb[bad[:3]]} oracle {ot[bad[:3]]}/{ob[bad[:3]]}")
    return ot, ob


def _inputs(rng, R, I, B=16, L_hi=4000, tie=False):
    L = rng.integers(0, L_hi, R).astype(np.int32)
    m = rng.integers(0, L_hi // B + 1, (R, I))
    m = np.minimum(m, (L // B)[:, None]).astype(np.int32)
    if tie:  # few distinct values: exact ties everywhere
        q = (rng.integers(0, 3, I) * 100).astype(np.int64)
        load = rng.integers(0, 3, I).astype(np.int32)
        m = (m // max(1, (L_hi // B) // 3) * max(1, (L_hi // B) // 3)).astype(np.int32)
    else:
        q = rng.integers(0, 10**6, I).astype(np.int64)
        load = rng.integers(0, 64, I).astype(np.int32)
    return m, L, q, load


@pytest.mark.parametrize("I", [1, 3, 64, 65, 257, 1000, 5000])
def test_random_parity(I):
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(8200 + I)
    R = 1200 if I <= 1000 else 200
    hits = {}
    for tie in (False, True):
        m, L, q, load = _inputs(rng, R, I, tie=tie)
        for kind in KINDS:
            for lam, rr in (((1, 2), 0), ((3, 4), 987654321), ((0, 7), 5), ((7, 7), 2**64 - 1), ((5, 9), 13)):
                if kind < oracle.SCORE_LINEAR and lam != (1, 2):
                    continue
                _, ob = _both(S, kind, m, L, q, load, 16, lam, rr)
                if kind == oracle.SCORE_HIT_FILTER:
                    hits[tie] = hits.get(tie, 0) + int((ob == 7).sum())
        # an idle cluster (every load 0) and the product's zero scores
        for kind in KINDS:
            _both(S, kind, m, L, q, np.zeros(I, np.int32), 16, (2, 3), 7)
    say(f"  I={I}: hit-filter decisions {hits}")
    assert all(v > 0 for v in hits.values())


def test_half_prompt_boundary_and_empty_prompts():
    """Holders at exactly half the prompt (not filtered) and one block above it (filtered),
    with B in {2, 256}; prompts of length 0 (hit ratio 0 by definition)."""
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(8301)
    for B in (2, 256):
        R, I = 600, 90
        L = (rng.integers(1, 40, R) * 2 * B).astype(np.int32)
        half = (L // (2 * B)).astype(np.int64)
        m = rng.integers(0, 2, (R, I)) * (half[:, None] + rng.integers(0, 2, (R, I)))
        m = np.minimum(m, (L // B)[:, None]).astype(np.int32)
        L[:60] = 0
        m[:60] = 0
        q = rng.integers(0, 10**4, I).astype(np.int64)
        load = rng.integers(0, 8, I).astype(np.int32)
        _, ob = _both(S, oracle.SCORE_HIT_FILTER, m, L, q, load, B, (1, 3), 11)
        assert (ob == 7).any() and (ob == 6).any()
        for kind in KINDS[:4]:
            _both(S, kind, m, L, q, load, B, (1, 3), 11)


def test_extremes_and_out_of_domain():
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(8401)
    R, I = 300, 130
    L = np.full(R, 1 << 24, np.int32)
    L[:80] = rng.integers(0, 1 << 24, 80)
    m = rng.integers(0, (1 << 24) // 256 + 1, (R, I))
    m = np.minimum(m, (L // 256)[:, None]).astype(np.int32)
    q = rng.integers((1 << 62) - 10**6, 1 << 62, I).astype(np.int64)
    load = rng.integers(2**31 - 1000, 2**31 - 1, I).astype(np.int32)
    for kind in KINDS:
        for lam in ((2**31 - 1, 2**31 - 1), (1, 2**31 - 1), (2**31 - 2, 2**31 - 1), (0, 1)):
            if kind < oracle.SCORE_LINEAR and lam != (0, 1):
                continue
            _both(S, kind, m, L, q, load, 256, lam, 2**64 - 1)
    # per-request domain errors: c above L / B, c negative, L negative, L above 2^24
    m2, L2 = m.copy(), L.copy()
    m2[3, 1] = L2[3] // 256 + 1
    m2[4, 7] = -1
    L2[5] = -1
    L2[6] = (1 << 24) + 1
    # per-instance domain errors make every request out of domain
    q_bad = q.copy()
    q_bad[9] = 1 << 62
    q_neg = q.copy()
    q_neg[0] = -1
    l_bad = load.copy()
    l_bad[129] = -1
    for kind in KINDS:
        _, ob = _both(S, kind, m2, L2, q, load, 256, (1, 2), 0)
        assert list(ob[3:7]) == [255] * 4 and (ob[7:] != 255).all()
        for qq, ll in ((q_bad, load), (q_neg, load), (q, l_bad)):
            _, ob = _both(S, kind, m, L, qq, ll, 256, (1, 2), 0)
            assert set(ob.tolist()) == {255}


def test_limits_and_host_errors():
    import torch
    from paper_2607_08565_amd import smetric as S
    rng = np.random.default_rng(8501)
    R, I = 24, 65536
    m, L, q, load = _inputs(rng, R, I, B=64)
    for kind in KINDS:
        _both(S, kind, m, L, q, load, 64, (2, 5), 40000)
    # empty batch
    e = torch.zeros((0, 5), dtype=torch.int32, device="cuda")
    t, b = S.route_score(oracle.SCORE_LOAD, e, to_dev(np.zeros(0, np.int32)), to_dev(np.zeros(5, np.int64)),
                         to_dev(np.zeros(5, np.int32)), 16)
    assert t.numel() == 0 and b.numel() == 0
    md, Ld, qd, ld = to_dev(m[:, :8].copy()), to_dev(L), to_dev(q[:8].copy()), to_dev(load[:8].copy())
    for kind, B, lam in ((5, 16, (0, 1)), (-1, 16, (0, 1)), (0, 3, (0, 1)), (0, 258, (0, 1)),
                         (oracle.SCORE_LINEAR, 16, (3, 2)), (oracle.SCORE_HIT_FILTER, 16, (0, 0)),
                         (oracle.SCORE_LINEAR, 16, (-1, 2))):
        with pytest.raises(S.SmetricError):
            S.route_score(kind, md, Ld, qd, ld, B, lam)
    # lam is ignored by the scorers that do not use it
    S.route_score(oracle.SCORE_TOKENS, md, Ld, qd, ld, 16, (0, 0))


def test_on_matched_rows_of_a_session_workload():
    """Every scorer on the real c rows of a scaled mid-fleet workload (closed loop: each
    batch's targets are inserted, so later turns see the sessions' own holders)."""
    from paper_2607_08565_amd import smetric as S
    wl = W.config1(n_sess=256, n_turns=3)
    pair = Pair(4_000_000, wl.n_inst)
    rng = np.random.default_rng(8601)
    prev = None
    for t in range(3):
        b = wl.batch(t, prev)
        d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(b.tokens, b.tok_off)
        gm = pair.gix.match(d_keys, d_boff, nb)
        om = pair.oix.match(okeys, blk_off)
        assert np.array_equal(gm.cpu().numpy(), om)
        qt = rng.integers(0, 20000, wl.n_inst).astype(np.int64)
        load = rng.integers(0, 30, wl.n_inst).astype(np.int32)
        counts = {}
        for kind in KINDS:
            ot, ob = _both(S, kind, om, b.prompt_len, qt, load, W.DEFAULT_PARAMS["block_size"], (9, 10), b.rr_base)
            counts[kind] = int((ob == 7).sum())
        say(f"  batch {t}: hit-filter decisions {counts[oracle.SCORE_HIT_FILTER]}")
        pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, ot, b.session, b.epoch)
        prev = ot
