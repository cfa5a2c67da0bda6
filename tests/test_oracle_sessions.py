"""Pins for the oracle's session reconstruction (App. A; CPU only).

The rule: a request follows an earlier request of the same user whose turn is smaller by
one and whose block-hash sequence its own starts with; chains form sessions.  Pins:
* hand-built traces covering each condition (user, turn + 1, prefix, most recent of
  several candidates, empty sequences, a gap of two turns, bad ranges);
* a hash-free brute force: with chained block keys, "key sequence of p is a prefix of
  r's" holds exactly when the full-block token prefix of p equals r's first tokens, so
  parents computed from tokens alone must match;
* the generator's ground truth: every parent is recovered except at compaction turns
  (whose rewritten prompt extends nothing), and every chain stays inside one true session.
"""
import numpy as np

import oracle
from paper_2607_08565_amd import workload as W

B = 16


def _run(prompts, user, turn):
    off = np.zeros(len(prompts) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    toks = np.concatenate([np.asarray(p, np.int32) for p in prompts]) if prompts else np.zeros(0, np.int32)
    blk_off, keys = oracle.hash_blocks(toks, off, B, W.DEFAULT_SEED)
    return oracle.sessions(keys, blk_off, user, turn)


def test_hand_built_trace():
    rng = np.random.default_rng(0)
    sysA, sysB = rng.integers(0, 1000, 32), rng.integers(0, 1000, 32)
    a0 = np.concatenate([sysA, rng.integers(0, 1000, 32)])      # user 0, session 1, turn 0
    a1 = np.concatenate([a0, rng.integers(0, 1000, 48)])        # its turn 1
    c0 = np.concatenate([sysA, rng.integers(0, 1000, 32)])      # user 0, session 2, turn 0 (same system prefix)
    c1 = np.concatenate([c0, rng.integers(0, 1000, 16)])
    b0 = np.concatenate([sysB, a0[32:]])                         # user 1: different prefix
    x1 = np.concatenate([a0, rng.integers(0, 1000, 16)])        # user 1 extending user 0's prompt: not linked
    a3 = np.concatenate([a1, rng.integers(0, 1000, 16)])        # user 0 turn 3: a gap of two turns
    prompts = [a0, c0, b0, a1, c1, x1, a3]
    user = [0, 0, 1, 0, 0, 1, 0]
    turn = [0, 0, 0, 1, 1, 1, 3]
    par, ses = _run(prompts, user, turn)
    assert par.tolist() == [-1, -1, -1, 0, 1, -1, -1]
    assert ses.tolist() == [0, 1, 2, 0, 1, 5, 6]


def test_most_recent_candidate_and_empty_sequences():
    rng = np.random.default_rng(1)
    p0 = rng.integers(0, 1000, 64)
    p1 = np.concatenate([p0, rng.integers(0, 1000, 32)])
    short = rng.integers(0, 1000, 10)  # no full block: the empty sequence
    prompts = [p0, p0, p1, short, p1, np.concatenate([p1, [1] * 16])]
    user = [7, 7, 7, 7, 7, 7]
    turn = [0, 0, 1, 1, 2, 2]
    par, ses = _run(prompts, user, turn)
    # request 2 has two candidates (0 and its retry 1): the most recent wins
    assert par[2] == 1
    # request 4 (turn 2): candidates at turn 1 are 2 (a prefix) and 3 (empty: a prefix of
    # anything) -> the most recent, 3
    assert par[4] == 3
    assert par[5] == 3
    # request 3 itself has no parent: the 4-block sequences of 0 and 1 are longer than its
    # empty one; it starts session 3, which 4 and 5 join
    assert par[3] == -1
    assert ses.tolist() == [0, 1, 1, 3, 3, 3]


def test_bad_ranges_are_skipped():
    keys = np.arange(1, 11, dtype=np.uint64)
    blk_off = np.array([0, 4, 3, 10], np.int64)  # request 1 has a negative range
    par, ses = oracle.sessions(keys, blk_off, [1, 1, 1], [0, 1, 2])
    assert par.tolist() == [-1, -1, -1] and ses.tolist() == [0, -1, 2]
    keys2 = np.arange(1, 9, dtype=np.uint64)
    par, ses = oracle.sessions(keys2, np.array([0, 4, 8], np.int64), [1, 1], [0, -1])
    assert par.tolist() == [-1, -1] and ses.tolist() == [0, -1]


def test_token_level_brute_force():
    """Parents from tokens alone (full-block token prefixes), no hashing."""
    for seed in range(6):
        tr = W.session_trace(n_users=6, sessions_per_user=3, turns=5, l0=96, prefix_len=48, app=(0, 40),
                             compact_len=40, p_compact=0.15, p_retry=0.1, seed=seed)
        R = tr.n_req
        blk_off, keys = oracle.hash_blocks(tr.tokens, tr.tok_off, B, W.DEFAULT_SEED)
        par, _ = oracle.sessions(keys, blk_off, tr.user, tr.turn)
        toks = [tr.tokens[tr.tok_off[r]:tr.tok_off[r + 1]] for r in range(R)]
        for r in range(R):
            want = -1
            for p in range(r - 1, -1, -1):
                if tr.user[p] != tr.user[r] or tr.turn[p] + 1 != tr.turn[r]:
                    continue
                n = (len(toks[p]) // B) * B  # tokens of p's full blocks
                if n <= (len(toks[r]) // B) * B and np.array_equal(toks[p][:n], toks[r][:n]):
                    want = p
                    break
            assert par[r] == want, (seed, r)


def test_recovers_the_generator_sessions():
    for seed in range(3):
        tr = W.session_trace(n_users=24, sessions_per_user=4, turns=6, seed=seed)
        blk_off, keys = oracle.hash_blocks(tr.tokens, tr.tok_off, B, W.DEFAULT_SEED)
        par, ses = oracle.sessions(keys, blk_off, tr.user, tr.turn)
        assert np.array_equal(par[~tr.compacted], tr.true_parent[~tr.compacted])
        assert (par[tr.compacted] == -1).all()
        # every reconstructed session lies inside one true session
        for s in np.unique(ses):
            assert len(np.unique(tr.true_session[ses == s])) == 1
