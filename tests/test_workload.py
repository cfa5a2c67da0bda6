"""Input generator checks (CPU only): determinism and the structural shapes each
configuration promises (append-only turns, shared prefixes, length ranges)."""
import numpy as np

from paper_2607_08565_amd import workload as W


def test_config0_shapes_and_append_only():
    wl = W.config0()
    assert wl.n_inst == 8 and wl.n_sess == 64 and wl.n_turns == 4
    assert np.all(wl.lens[0] == 1024)
    d = np.diff(wl.lens, axis=0)
    assert d.min() >= 128 and d.max() <= 1024
    b2 = wl.batch(2)
    b3 = wl.batch(3)
    for s in range(wl.n_sess):
        p2 = b2.tokens[b2.tok_off[s]: b2.tok_off[s + 1]]
        p3 = b3.tokens[b3.tok_off[s]: b3.tok_off[s + 1]]
        assert np.array_equal(p3[: len(p2)], p2)
    firsts = np.array([b2.tokens[b2.tok_off[s]: b2.tok_off[s] + 512] for s in range(64)])
    shared = [s for s in range(64) if np.array_equal(firsts[s], firsts[np.argmax([np.array_equal(firsts[s], f) for f in firsts])])]
    n_with_prefix = max(sum(np.array_equal(firsts[s], firsts[t]) for t in range(64)) for s in range(64))
    assert n_with_prefix == 16 and shared
    assert b3.q.min() >= 0 and b3.q.max() <= 100 * W.Q_UNIT_NS and b3.hist_len.tolist() == wl.lens[2].tolist()


def test_determinism():
    a = W.config0().batch(1)
    b = W.config0().batch(1)
    assert np.array_equal(a.tokens, b.tokens) and np.array_equal(a.q, b.q)


def test_throughput_batch_structure():
    tw = W.ThroughputWorkload(n_req=256, n_inst=64)
    tb = tw.batch(0)
    L = tb.batch.prompt_len.astype(np.int64)
    assert L.min() >= 1024 and L.max() <= 131072
    assert np.all(tb.prior_len == 16 * np.floor(0.7 * (L // 16)))
    for r in range(256):
        p = tb.batch.tokens[tb.batch.tok_off[r]: tb.batch.tok_off[r + 1]]
        pre = tw.prefixes[tb.prefix_of[r]]
        n = min(len(pre), len(p))
        assert np.array_equal(p[:n], pre[:n])
    assert np.all(tb.batch.turn == 1) and np.all(tb.batch.hist_len == tb.prior_len)
    k, i, s = tw.filler(1000)
    assert k.min() >= 1 and i.max() < 64
