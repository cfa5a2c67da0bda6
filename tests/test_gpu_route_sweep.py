"""GPU route rules (through the C ABI) vs the CPU oracle, bit for bit, on seeded random
batches that vary everything at once: instance counts around the 64-lane wave and the
1,024-instance register rows, block sizes 2..256, prompt lengths up to 2^24 tokens (and
empty prompts), hit rows from none to whole prompts (one instance holding most of a prompt,
an out-of-domain hit), loads from a few queued requests to just under 2^62 ns, every cost
and SLO parameter from 0 to its 2^32 limit, SLACK from 0 to unbounded, and 64-bit
round-robin bases.  The batch rule and its colocation variant, both online rules (final
loads and request counts included), and the five comparison scorers with a random lam; a
batch the online rules cannot take within their 128-bit bound is refused with EINVAL on
both sides of the check."""
import numpy as np
import pytest

import oracle
from paper_2607_08565_amd import workload as W
from tests.parity import to_dev

pytestmark = pytest.mark.gpu

INSTANCES = [1, 2, 3, 63, 64, 65, 127, 128, 129, 511, 512, 513, 1000, 1024, 1025, 2047, 2048, 3000, 4096]


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _case(seed):
    rng = np.random.default_rng(seed)
    I = int(rng.choice(INSTANCES))
    R = int(rng.integers(0, 2500 if I <= 1024 else 600))
    B = int(rng.choice([2, 4, 16, 16, 16, 64, 256]))
    l_hi = int(rng.choice([64, 4000, 40000, 1 << 20, 1 << 24]))
    L = rng.integers(0, l_hi + 1, R).astype(np.int32)
    if R and rng.random() < 0.3:
        L[rng.random(R) < 0.2] = 0
    m = (rng.random((R, I)) * rng.random() * (L // B + 1)[:, None]).astype(np.int32)
    m = np.minimum(m, (L // B)[:, None]).astype(np.int32)
    if R and rng.random() < 0.3:  # rows cached mostly on one instance
        prev = rng.integers(0, I, R)
        m[np.arange(R), prev] = (L // B) * rng.integers(50, 101, R) // 100
    if R and rng.random() < 0.2:  # one request out of domain (c > L / B)
        m[rng.integers(0, R), rng.integers(0, I)] = 1 << 24
    hist = rng.integers(0, l_hi + 1, R).astype(np.int32)
    turn = rng.integers(0, 3, R).astype(np.int32)
    q = [rng.integers(0, 200, I) * W.Q_UNIT_NS, rng.integers(0, 1 << 40, I),
         rng.integers((1 << 49) - (1 << 40), 1 << 49, I), rng.integers(0, 1 << 62, I)][int(rng.integers(0, 4))]
    q = q.astype(np.int64)
    lim = 1 << 32
    p = dict(W.DEFAULT_PARAMS, block_size=B,
             c_lin=int(rng.choice([0, 1, 100000, 1 << 20, lim])), c_att=int(rng.choice([0, 1, 3, 1 << 12, lim])),
             slo_b=int(rng.choice([0, 10**9, lim])), slo_a=int(rng.choice([0, 62500, lim])),
             slack_num=int(rng.choice([0, 1, 3, 1 << 20])), slack_den=int(rng.choice([0, 1, 2, 7])),
             hit_num=int(rng.choice([0, 1, 3])), hit_den=int(rng.choice([4, 5, 7])))
    rr = int(rng.integers(0, 1 << 63))
    slack = np.where(rng.random(I) < 0.3, oracle.NO_DECODE, rng.integers(-10**9, 10**10, I)).astype(np.int64)
    n_run = rng.integers(0, 50, I).astype(np.int32)
    return m, L, hist, turn, q, slack, n_run, p, rr


def _same(R, got, want):
    return all(np.array_equal(g.cpu().numpy()[:len(w)] if g.dim() else g.cpu().numpy(), w) for g, w in zip(got, want))


@pytest.mark.parametrize("chunk", range(4))
def test_route_rules_on_random_batches(chunk):
    from paper_2607_08565_amd import smetric as S
    for seed in range(91000 + 40 * chunk, 91000 + 40 * (chunk + 1)):
        m, L, hist, turn, q, slack, n_run, p, rr = _case(seed)
        R, I = m.shape
        args = (to_dev(m), to_dev(L), to_dev(hist), to_dev(turn), to_dev(q))
        assert _same(R, S.route(*args, p, rr), oracle.route(m, L, hist, turn, q, p, rr)), f"route, seed {seed}"
        assert _same(R, S.route_coloc(*args, to_dev(slack), to_dev(n_run), p, rr),
                     oracle.route_coloc(m, L, hist, turn, q, slack, n_run, p, rr)), f"route_coloc, seed {seed}"
        _online(S.route_seq, oracle.route_seq, (args, (m, L, hist, turn, q)), (), p, rr, R, f"route_seq, seed {seed}")
        _online(S.route_seq_coloc, oracle.route_seq_coloc, (args, (m, L, hist, turn, q)),
                ((to_dev(slack), to_dev(n_run)), (slack, n_run)), p, rr, R, f"route_seq_coloc, seed {seed}")
        lam_den = 1 + seed % 97
        lam = ((seed * 7) % (lam_den + 1), lam_den)
        for kind in range(5):
            assert _same(R, S.route_score(kind, args[0], args[1], args[4], to_dev(n_run), p["block_size"], lam, rr),
                         oracle.route_score(kind, m, L, q, n_run, p["block_size"], lam, rr)), \
                f"route_score kind {kind}, seed {seed}"


def _online(gpu_fn, oracle_fn, base, extra, p, rr, R, what):
    """Both sides decide the batch, or both refuse it (outside the 128-bit bound)."""
    from paper_2607_08565_amd import smetric as S
    g_args = base[0] + (extra[0] if extra else ())
    o_args = base[1] + (extra[1] if extra else ())
    try:
        got = gpu_fn(*g_args, p, rr)
    except S.SmetricError:
        got = None
    try:
        want = oracle_fn(*o_args, p, rr)
    except ValueError:
        want = None
    assert (got is None) == (want is None), f"{what}: refused on one side only"
    if got is not None:
        assert _same(R, got, want), what
