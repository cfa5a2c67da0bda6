"""Prompts whose chained block keys land on the index's reserved markers.

A block key is F(s_j), with F the SplitMix64 finaliser and s_j the affine chain state
(Sec. 3.1 / App. A chained block hashes, reading SMH64-v1).  F maps 0 to 0, and both 0
and 2^64-1 are the device table's EMPTY and TOMB markers, so the definition remaps a
key of 0 to 1 and a key of 2^64-1 to 2^64-2.  Random prompts reach those values with
probability 2^-63 per block; these prompts reach them on purpose:

  * the wanted chain state is s = F^-1(0) = 0 or F^-1(2^64-1);
  * the block's innovation must be e = s - M s_prev (mod 2^64);
  * the digest must be d = F^-1(e) - j (the position salt);
  * the NH digest sum_k a_k b_k (a_k = x_2k + K_2k, b_k = x_2k+1 + K_2k+1, mod 2^32)
    is solved with d = hi 2^32 + lo: (2^32 - 1) hi + 1 lo + 1 hi = d, every later pair
    given a_k = 0 (its second token stays random).

F^-1 undoes F's three invertible steps (two xor-shifts and two odd multiplies); its
round trip is pinned against published SplitMix64 output in the hash tests.  Only the
constants K, M and s_init come from the oracle (pinned to the SplitMix64 stream); the
state of a random block that precedes a constructed one is read back from the oracle's
key for it (F^-1 of an unreserved key), so a wrong chain anywhere makes the constructed
block miss its marker and the test that uses it fail.
"""
from __future__ import annotations

import numpy as np

import oracle

MASK = (1 << 64) - 1
U32 = (1 << 32) - 1
KEY_EMPTY = 0
KEY_TOMB = MASK


def _inv_xorshift(y: int, s: int) -> int:
    z = y
    for _ in range(64 // s + 1):
        z = y ^ (z >> s)
    return z & MASK


def inv_finaliser(y: int) -> int:
    """Inverse of the SplitMix64 output function."""
    z = _inv_xorshift(y, 31)
    z = (z * pow(0x94D049BB133111EB, -1, 1 << 64)) & MASK
    z = _inv_xorshift(z, 27)
    z = (z * pow(0xBF58476D1CE4E5B9, -1, 1 << 64)) & MASK
    z = _inv_xorshift(z, 30)
    return z


def block_for_state(K, M: int, s_prev: int, j: int, s_want: int, rng: np.random.Generator) -> np.ndarray:
    """B tokens (int32 bit patterns) that take the chain from s_prev to s_want at block j."""
    B = len(K)
    assert B % 2 == 0 and B >= 6, "three token pairs carry the digest"
    e = (s_want - M * s_prev) & MASK
    d = (inv_finaliser(e) - j) & MASK
    hi, lo = d >> 32, d & U32
    a = [U32, 1, 1] + [0] * (B // 2 - 3)
    b = [hi, lo, hi] + [int(v) for v in rng.integers(0, 1 << 32, B // 2 - 3, dtype=np.uint64)]
    x = np.zeros(B, np.uint32)
    for k in range(B // 2):
        x[2 * k] = (a[k] - int(K[2 * k])) & U32
        x[2 * k + 1] = (b[k] - int(K[2 * k + 1])) & U32
    return x.view(np.int32)


def prompt_with_reserved(n_blocks: int, marks: dict[int, int], seed: int, B: int = 16, tail: int = 0,
                         rng: np.random.Generator | None = None) -> np.ndarray:
    """A prompt of n_blocks full blocks (+ `tail` extra tokens) whose block j, for each
    j in marks, has the unremapped key marks[j] (KEY_EMPTY or KEY_TOMB); every other block
    is random int32 bit patterns."""
    rng = rng or np.random.default_rng(seed & 0xFFFF)
    K, M, s_init = oracle.hash_consts(seed, B)
    toks = []
    s_prev = s_init
    for j in range(n_blocks):
        if j in marks:
            s = inv_finaliser(marks[j])
            toks.append(block_for_state(K, M, s_prev, j, s, rng))
            s_prev = s
        else:
            blk = rng.integers(-2**31, 2**31 - 1, B, dtype=np.int64).astype(np.int32)
            toks.append(blk)
            _, keys = oracle.hash_blocks(np.concatenate(toks), [0, B * (j + 1)], B, seed)
            k = int(keys[j])
            assert k not in (1, MASK - 1), "a random block hit a remapped value"
            s_prev = inv_finaliser(k)
    toks.append(rng.integers(-2**31, 2**31 - 1, tail, dtype=np.int64).astype(np.int32))
    return np.concatenate(toks)
