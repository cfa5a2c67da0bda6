"""GPU session reconstruction (App. A, through the C ABI) vs the CPU oracle, bit for bit:
parent and session of every request.  Traces with many sessions per user sharing a
system prefix, compactions, retries (several candidate parents), prompts shorter than a
block (empty sequences), prompts longer than one wavefront's 64 prefix lengths, and bad
inputs."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_08565_amd import workload as W
from tests.parity import say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _gpu_keys(S, tokens, tok_off):
    blk_off, nb = S.block_offsets(tok_off)
    keys = S.hash_blocks(to_dev(tokens if len(tokens) else np.zeros(1, np.int32)), to_dev(tok_off), to_dev(blk_off), nb)
    return keys, blk_off, nb


def _check(S, tr_tokens, tr_off, user, turn):
    keys, blk_off, nb = _gpu_keys(S, tr_tokens, tr_off)
    ob, ok = oracle.hash_blocks(tr_tokens, tr_off, 16, W.DEFAULT_SEED)
    assert np.array_equal(keys[:nb].cpu().numpy(), ok)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    gp, gs = S.sessions(keys, to_dev(blk_off), nb, to_dev(np.asarray(user, np.uint32)),
                        to_dev(np.asarray(turn, np.int32)), status=status)
    op, os_ = oracle.sessions(ok, ob, user, turn)
    gp, gs = gp.cpu().numpy(), gs.cpu().numpy()
    assert np.array_equal(gp, op), f"parents differ at {np.nonzero(gp != op)[0][:5]}"
    assert np.array_equal(gs, os_), f"sessions differ at {np.nonzero(gs != os_)[0][:5]}"
    return op, os_, int(status.item())


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_traces(seed):
    from paper_2607_08565_amd import smetric as S
    tr = W.session_trace(n_users=40, sessions_per_user=5, turns=7, p_compact=0.1, p_retry=0.1, seed=seed)
    op, os_, st = _check(S, tr.tokens, tr.tok_off, tr.user, tr.turn)
    assert st == 0
    say(f"  {tr.n_req} requests, {int((op >= 0).sum())} linked, {len(np.unique(os_))} sessions")


def test_short_prompts_and_single_user():
    """One user, many sessions with identical prefixes; prompts of 0-40 tokens (often no
    full block), so empty sequences are parents of everything one turn later."""
    from paper_2607_08565_amd import smetric as S
    tr = W.session_trace(n_users=1, sessions_per_user=60, turns=6, l0=24, prefix_len=16, app=(0, 12),
                         compact_len=8, p_compact=0.2, p_retry=0.2, seed=5)
    _check(S, tr.tokens, tr.tok_off, tr.user, tr.turn)


def test_long_prompts_many_prefix_lengths():
    """Prompts of thousands of blocks: every wavefront walks many 64-length rounds."""
    from paper_2607_08565_amd import smetric as S
    tr = W.session_trace(n_users=4, sessions_per_user=3, turns=4, l0=40_000, prefix_len=20_000, app=(2000, 9000),
                         seed=7)
    op, _, _ = _check(S, tr.tokens, tr.tok_off, tr.user, tr.turn)
    assert (op >= 0).sum() > 0


def test_bad_inputs_flag_status():
    from paper_2607_08565_amd import smetric as S
    tr = W.session_trace(n_users=3, sessions_per_user=2, turns=3, l0=64, prefix_len=32, app=(16, 48), seed=9)
    keys, blk_off, nb = _gpu_keys(S, tr.tokens, tr.tok_off)
    bad = blk_off.copy()
    bad[2] = bad[3] + 1  # request 2 gets a negative range (and request 1 a longer one)
    turn = tr.turn.copy()
    turn[4] = -3
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    gp, gs = S.sessions(keys, to_dev(bad), nb, to_dev(tr.user), to_dev(turn), status=status)
    op, os_ = oracle.sessions(keys[:nb].cpu().numpy(), bad, tr.user, turn)
    assert np.array_equal(gp.cpu().numpy(), op) and np.array_equal(gs.cpu().numpy(), os_)
    assert int(status.item()) == oracle.EINVAL
    assert op[2] == -1 and os_[2] == -1 and op[4] == -1 and os_[4] == -1


def test_tiny_batches():
    from paper_2607_08565_amd import smetric as S
    for prompts, user, turn in (([[1] * 40], [3], [2]), ([[1] * 40, [1] * 56], [3, 3], [0, 1]),
                                ([[], [5] * 16], [1, 1], [0, 1])):
        toks = np.concatenate([np.asarray(p, np.int32) for p in prompts])
        off = np.zeros(len(prompts) + 1, np.int64)
        off[1:] = np.cumsum([len(p) for p in prompts])
        _check(S, toks, off, np.asarray(user, np.uint32), np.asarray(turn, np.int32))


def test_random_trace_shapes():
    """Seeded random trace shapes: 1-59 users, 1-7 sessions each, 1-8 turns, prompts from
    empty to thousands of tokens, no or short or long shared prefixes, compactions and
    retries from never to often."""
    from paper_2607_08565_amd import smetric as S
    for case in range(60000, 60030):
        rng = np.random.default_rng(case)
        tr = W.session_trace(n_users=int(rng.integers(1, 60)), sessions_per_user=int(rng.integers(1, 8)),
                             turns=int(rng.integers(1, 9)), l0=int(rng.choice([0, 8, 24, 300, 2048])),
                             prefix_len=int(rng.choice([0, 16, 100, 1024])),
                             app=tuple(sorted(rng.integers(0, 3000, 2).tolist())),
                             p_compact=float(rng.choice([0, 0.05, 0.3])), p_retry=float(rng.choice([0, 0.03, 0.3])),
                             compact_len=int(rng.choice([0, 8, 1024])), seed=case)
        _check(S, tr.tokens, tr.tok_off, tr.user, tr.turn)
