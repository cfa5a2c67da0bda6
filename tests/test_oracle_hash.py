"""Pins for the oracle's block split and chained block keys (CPU only).

The paper fixes no hash function: it measures reuse at KV$-block granularity and
identifies a prompt prefix by its sequence of chained block hashes (Sec. 3.1, App. A).
These tests pin the oracle's hash by what does not depend on retyping its formula:
published SplitMix64 output for the constants, and structural identities recovered by
*inverting* the SplitMix64 finaliser (the affine chain, the position salt and the
bilinear pairing of the NH digest), plus the prefix/sensitivity properties the paper
relies on.
"""
import os

import numpy as np
import pytest

import oracle

MASK = (1 << 64) - 1
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _inv_xorshift(y: int, s: int) -> int:
    # inverse of z -> z ^ (z >> s) on 64 bits
    z = y
    for _ in range(64 // s + 1):
        z = y ^ (z >> s)
    return z & MASK


def inv_finaliser(y: int) -> int:
    """Inverse of the SplitMix64 output function, from its three invertible steps."""
    z = _inv_xorshift(y, 31)
    z = (z * pow(0x94D049BB133111EB, -1, 1 << 64)) & MASK
    z = _inv_xorshift(z, 27)
    z = (z * pow(0xBF58476D1CE4E5B9, -1, 1 << 64)) & MASK
    z = _inv_xorshift(z, 30)
    return z


def chain_states(keys):
    return [inv_finaliser(int(k)) for k in keys]


def test_splitmix64_published_vector():
    want = [int(x) for x in open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt")) if x.strip() and not x.startswith("#")]
    assert oracle.splitmix_stream(1234567, 5) == want


def test_inverse_finaliser_roundtrip():
    # the finaliser of output 1 for seed 1234567 applied to state seed + golden increment
    st = (1234567 + 0x9E3779B97F4A7C15) & MASK
    assert inv_finaliser(oracle.splitmix_stream(1234567, 1)[0]) == st


@pytest.mark.parametrize("B", [2, 16, 64])
def test_constants_are_the_splitmix_stream(B):
    seed = 0x1234_5678_9ABC_DEF0
    K, M, s0 = oracle.hash_consts(seed, B)
    out = oracle.splitmix_stream(seed, B + 2)
    assert [int(k) for k in K] == [o & 0xFFFFFFFF for o in out[:B]]
    assert M == out[B] | 1 and M & 1
    assert s0 == out[B + 1]


def _keys(tokens, B=16, seed=7):
    tokens = np.asarray(tokens, np.int32)
    _, keys = oracle.hash_blocks(tokens, [0, len(tokens)], B, seed)
    return [int(k) for k in keys]


def test_block_split_counts_only_full_blocks():
    rng = np.random.default_rng(1)
    t = rng.integers(0, 151936, 100, dtype=np.int32)
    off = [0, 15, 31, 63, 63, 100]  # lengths 15, 16, 32, 0, 37
    blk_off, keys = oracle.hash_blocks(t, off, 16, 3)
    assert list(blk_off) == [0, 0, 1, 3, 3, 5]
    assert len(keys) == 5


def test_affine_chain_innovation_depends_only_on_block_and_position():
    """s_j - M s_{j-1} must equal F(d_j + j), a function of block j's tokens and j only."""
    B, seed = 16, 99
    _, M, s0 = oracle.hash_consts(seed, B)
    rng = np.random.default_rng(2)
    blk = rng.integers(0, 151936, B, dtype=np.int32)
    h1 = rng.integers(0, 151936, 3 * B, dtype=np.int32)
    h2 = rng.integers(0, 151936, 3 * B, dtype=np.int32)
    s1 = chain_states(_keys(np.concatenate([h1, blk]), B, seed))
    s2 = chain_states(_keys(np.concatenate([h2, blk]), B, seed))
    e1 = (s1[3] - M * s1[2]) & MASK
    e2 = (s2[3] - M * s2[2]) & MASK
    assert e1 == e2
    # the chain starts from s_init: block 0's innovation is s_0 - M s_init, same for any tail
    a = chain_states(_keys(np.concatenate([blk, h1]), B, seed))
    b = chain_states(_keys(np.concatenate([blk, h2]), B, seed))
    assert a[0] == b[0]
    assert ((a[0] - M * s0) & MASK) == ((b[0] - M * s0) & MASK)
    # the same block at another position gets another innovation (position salt)
    e_pos0 = (a[0] - M * s0) & MASK
    assert e_pos0 != e1
    # and recovering d_j + j: innovation -> F^-1 gives d_j + j, so d_j is position-free
    d_at3 = (inv_finaliser(e1) - 3) & MASK
    d_at0 = (inv_finaliser(e_pos0) - 0) & MASK
    assert d_at3 == d_at0


def _digest(block, B=16, seed=5, M=None, s0=None):
    """d_j recovered from the oracle for a single-block prompt: F^-1(F^-1(key) - M s_init)."""
    _, M, s0 = oracle.hash_consts(seed, B)
    (k,) = _keys(block, B, seed)
    s = inv_finaliser(k)
    return inv_finaliser((s - M * s0) & MASK)  # = d + 0


def test_nh_digest_is_bilinear_in_adjacent_token_pairs():
    """Raising token 2k by one adds (x[2k+1] + K[2k+1]) mod 2^32 to the digest, and
    raising token 2k+1 adds (x[2k] + K[2k]) mod 2^32: pairs are (2k, 2k+1), each offset by
    its own constant, products summed mod 2^64."""
    B, seed = 16, 5
    K, _, _ = oracle.hash_consts(seed, B)
    rng = np.random.default_rng(3)
    for _ in range(4):
        x = rng.integers(0, 151936, B, dtype=np.int64)
        base = _digest(x.astype(np.int32), B, seed)
        for k in range(B // 2):
            for pos, other in ((2 * k, 2 * k + 1), (2 * k + 1, 2 * k)):
                if (int(x[pos]) + int(K[pos])) & 0xFFFFFFFF == 0xFFFFFFFF:
                    continue  # +1 would wrap the 32-bit offset sum
                y = x.copy()
                y[pos] += 1
                got = (_digest(y.astype(np.int32), B, seed) - base) & MASK
                assert got == (int(x[other]) + int(K[other])) & 0xFFFFFFFF, (k, pos)


def test_prefix_property_and_sensitivity():
    rng = np.random.default_rng(4)
    t = rng.integers(0, 151936, 40 * 16 + 7, dtype=np.int32)
    full = _keys(t)
    for L in (0, 15, 16, 17, 100, 320, 639):
        assert _keys(t[:L]) == full[: L // 16]
    # changing one token changes every key from its block on and no key before it
    for pos in (0, 15, 16, 200, 40 * 16 - 1):
        u = t.copy()
        u[pos] ^= 1
        k2 = _keys(u)
        b = pos // 16
        assert k2[:b] == full[:b]
        assert all(a != c for a, c in zip(k2[b:], full[b:]))


def test_shared_prefix_gives_equal_keys_until_divergence():
    rng = np.random.default_rng(5)
    pre = rng.integers(0, 151936, 512 + 5, dtype=np.int32)
    a = np.concatenate([pre, rng.integers(0, 151936, 300, dtype=np.int32)])
    b = np.concatenate([pre, rng.integers(0, 151936, 300, dtype=np.int32)])
    ka, kb = _keys(a), _keys(b)
    n_shared = len(pre) // 16
    assert ka[:n_shared] == kb[:n_shared]
    assert all(x != y for x, y in zip(ka[n_shared:], kb[n_shared:]))


def test_seed_and_block_size_change_keys():
    rng = np.random.default_rng(6)
    t = rng.integers(0, 151936, 64, dtype=np.int32)
    assert _keys(t, 16, 1) != _keys(t, 16, 2)
    assert len(_keys(t, 32, 1)) == 2


def test_keys_never_reserved_and_no_collisions():
    rng = np.random.default_rng(7)
    t = rng.integers(0, 151936, 200_000, dtype=np.int32)
    off = np.arange(0, 200_001, 1000)
    _, keys = oracle.hash_blocks(t, off, 16, 11)
    assert len(np.unique(keys)) == len(keys)
    assert not np.any(keys == 0) and not np.any(keys == np.uint64(MASK))
    # bit balance: every key bit is set in roughly half of the keys
    bits = ((keys[:, None] >> np.arange(64, dtype=np.uint64)) & np.uint64(1)).mean(axis=0)
    assert np.all(np.abs(bits - 0.5) < 0.05)


def test_bad_block_size_rejected():
    with pytest.raises(ValueError):
        oracle.hash_blocks(np.zeros(10, np.int32), [0, 10], 15, 0)


# --- the reserved-marker remap (last step of the chained block key) ------------------
# Keys 0 and 2^64-1 are the device table's EMPTY and TOMB markers; the definition sends
# them to 1 and 2^64-2.  The prompts below are built (tests/reserved_keys.py) so that
# their unremapped key is exactly a marker.

from tests.reserved_keys import KEY_EMPTY, KEY_TOMB, prompt_with_reserved  # noqa: E402


@pytest.mark.parametrize("B", [16, 8, 64])
def test_remap_sends_markers_to_their_neighbours(B):
    seed = 0x5EED
    for marker, want in ((KEY_EMPTY, 1), (KEY_TOMB, MASK - 1)):
        t = prompt_with_reserved(1, {0: marker}, seed, B)
        _, keys = oracle.hash_blocks(t, [0, len(t)], B, seed)
        assert [int(k) for k in keys] == [want], (B, hex(marker))


def test_remap_does_not_feed_back_into_the_chain():
    """The chain continues from the true state s_j (0, or F^-1(2^64-1)), not from the
    remapped key: block j+1's state equals its innovation plus M s_j, and the innovation
    is recovered from the same block at the same position after an ordinary history."""
    B, seed = 16, 31
    _, M, _ = oracle.hash_consts(seed, B)
    rng = np.random.default_rng(8)
    nxt = rng.integers(0, 151936, B, dtype=np.int32)
    other = rng.integers(0, 151936, B, dtype=np.int32)
    ko = _keys(np.concatenate([other, nxt]), B, seed)
    innov = (inv_finaliser(ko[1]) - M * inv_finaliser(ko[0])) & MASK
    for marker in (KEY_EMPTY, KEY_TOMB):
        t = np.concatenate([prompt_with_reserved(1, {0: marker}, seed, B), nxt])
        k = _keys(t, B, seed)
        s0 = inv_finaliser(marker)
        assert k[0] in (1, MASK - 1)
        assert inv_finaliser(k[1]) == (M * s0 + innov) & MASK


def test_remap_in_the_middle_of_a_prompt():
    """A marker key at block 5 of 9 and at the last block: only those keys move, and the
    keys after block 5 are those of the unremapped chain (the same prompt's prefix
    property holds through it)."""
    B, seed = 16, 77
    t = prompt_with_reserved(9, {5: KEY_TOMB, 8: KEY_EMPTY}, seed, B, tail=11)
    k = _keys(t, B, seed)
    assert k[5] == MASK - 1 and k[8] == 1
    assert all(v not in (0, MASK, 1, MASK - 1) for i, v in enumerate(k) if i not in (5, 8))
    for L in (5 * B, 6 * B, 6 * B + 3, 9 * B):
        assert _keys(t[:L], B, seed) == k[: L // B]
