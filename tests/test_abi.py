"""The C-ABI library loads on the CPU and exports every entry point include/*.h declares
(no GPU work is launched)."""
import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"^\s*(?:int|void|uint64_t|int32_t)\s+(smetric_\w+)\s*\(", text, flags=re.M))
    return sorted(names)


def test_header_declares_the_hot_path_calls():
    names = declared_symbols()
    for must in ("smetric_hash_blocks", "smetric_match", "smetric_route", "smetric_index_insert",
                 "smetric_index_evict"):
        assert must in names


def test_library_exports_every_declared_symbol():
    from paper_2607_08565_amd import smetric as S
    lib = ctypes.CDLL(S.LIB_PATH)
    missing = [n for n in declared_symbols() if not hasattr(lib, n)]
    assert not missing, missing
    assert set(S.EXPORTED) == set(declared_symbols())


def test_host_side_errors_without_gpu():
    from paper_2607_08565_amd import smetric as S
    assert S.version() >= 1
    with pytest.raises(S.SmetricError):
        S.index_bytes(0, 8)
    with pytest.raises(S.SmetricError):
        S.index_bytes(100, 65537)
    # an explicit slot count: whole 8-slot buckets, at least 1/16 free at capacity
    # (capacity 1,000,000 over 1,024 instances keeps 3,906 bitmap records of T = 8 slots)
    reserved = 1_000_000 + 8 * 3906
    assert S.index_bytes(1_000_000, 1024, 2**21) > 16 * 2**21
    assert S.index_bytes(1_000_000, 1024, 1_120_000) < S.index_bytes(1_000_000, 1024)  # fuller than the default
    lo = -(-reserved * 16 // 15)
    S.index_bytes(1_000_000, 1024, lo + 8)
    with pytest.raises(S.SmetricError):
        S.index_bytes(1_000_000, 1024, lo - 16)
    with pytest.raises(S.SmetricError):
        S.index_bytes(100, 8, 2**41 + 1)
    with pytest.raises(S.SmetricError):
        S.block_offsets([0, 10], 15)
    blk, nb = S.block_offsets([0, 15, 31, 100, 100], 16)
    assert blk.tolist() == [0, 0, 1, 5, 5] and nb == 5
    assert S.insert_ws_bytes(1000) > 16 * 1000
    # the online colocation route's workspace: records per request, two blocks of candidate
    # lists, two copies of the instance state; at most 4,096 instances
    small, big = S.route_seq_coloc_ws_bytes(1, 8), S.route_seq_coloc_ws_bytes(16384, 1024)
    assert big >= 16384 * 48 + 2 * 1024 * 20 > small > 0 and small % 256 == 0 and big % 256 == 0
    assert S.route_seq_coloc_ws_bytes(0, 4096) > 2 * 4096 * 20
    for bad in ((-1, 8), (10, 0), (10, 4097)):
        with pytest.raises(S.SmetricError):
            S.route_seq_coloc_ws_bytes(*bad)


def test_route_score_host_checks_without_gpu():
    """smetric_route_score rejects bad scalars on the host, before any launch, and an empty
    batch returns at once (nothing is enqueued, so no GPU is needed)."""
    from paper_2607_08565_amd import smetric as S
    f = S._lib.smetric_route_score
    call = lambda kind, n_req, I, B, lam: f(kind, None, n_req, I, None, None, None, B, lam[0], lam[1], 0, None, None,
                                           None)
    assert call(0, 0, 8, 16, (0, 0)) == S.OK                   # empty batch; lam unused by kind 0
    assert call(3, 0, 8, 16, (1, 2)) == S.OK
    for args in ((5, 0, 8, 16, (0, 1)), (-1, 0, 8, 16, (0, 1)), (0, -1, 8, 16, (0, 1)), (0, 0, 0, 16, (0, 1)),
                 (0, 0, 65537, 16, (0, 1)), (0, 0, 8, 3, (0, 1)), (0, 0, 8, 258, (0, 1)), (3, 0, 8, 16, (2, 1)),
                 (4, 0, 8, 16, (0, 0)), (3, 0, 8, 16, (-1, 2))):
        assert call(*args) == S.EINVAL, args
    assert call(1, 4, 8, 16, (0, 1)) == S.EINVAL               # null device pointers
