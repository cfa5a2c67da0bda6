"""The allocation-free online route (smetric_route_seq_noalloc) against the same route
with a caller workspace (smetric_route_seq), through the C ABI: bit for bit on targets,
branches and final loads, on two calls in a row -- the second smaller, so it runs over
the first call's leftover records -- and the size limit's error."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2607_08565_amd import workload as W
from tests.parity import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _batch(rng, R, I):
    """Route inputs shaped like a batch of follow-ups: each request's prior turn on one
    instance (70 % of its blocks), a few partial hits elsewhere, some first turns."""
    L = rng.integers(1024, 65536, R).astype(np.int32)
    hist = (L // 16 * 7 // 10 * 16).astype(np.int32)
    turn = (rng.random(R) > 0.1).astype(np.int32)
    m = np.zeros((R, I), np.int32)
    prev = rng.integers(0, I, R)
    m[np.arange(R), prev] = np.where(turn > 0, hist // 16, 0)
    for _ in range(3):
        j = rng.integers(0, I, R)
        m[np.arange(R), j] = np.maximum(m[np.arange(R), j], rng.integers(0, 64, R))
    q = rng.poisson(50, I).astype(np.int64) * 20_000_000
    return m, L, hist, turn, q


def _both(m, L, hist, turn, q, rr_base):
    from paper_2607_08565_amd import smetric as S
    R, I = m.shape
    d = [to_dev(x) for x in (m, L, hist, turn, q)]
    t1, b1, q1 = S.route_seq(*d, W.DEFAULT_PARAMS, rr_base)
    t2 = torch.full((R,), -7, dtype=torch.int32, device="cuda")
    b2 = torch.full((R,), 77, dtype=torch.uint8, device="cuda")
    q2 = torch.full((I,), -7, dtype=torch.int64, device="cuda")
    S.route_seq_noalloc(*d, W.DEFAULT_PARAMS, rr_base, t2, b2, q2)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in (t1, b1, q1, t2, b2, q2)]


def test_noalloc_route_equals_the_workspace_route_twice():
    rng = np.random.default_rng(71)
    first = _batch(rng, 5000, 512)
    t1, b1, q1, t2, b2, q2 = _both(*first, rr_base=11)
    assert np.array_equal(t1, t2) and np.array_equal(b1, b2) and np.array_equal(q1, q2)
    assert len(np.unique(b1)) >= 3  # sticks, last resorts / migrations and first turns
    # a smaller second call: the scratch still holds the first call's records past its end
    second = _batch(rng, 1200, 300)
    t1, b1, q1, t2, b2, q2 = _both(*second, rr_base=5)
    assert np.array_equal(t1, t2) and np.array_equal(b1, b2) and np.array_equal(q1, q2)
    # and an empty one
    from paper_2607_08565_amd import smetric as S
    e = _batch(rng, 0, 64)
    t1, b1, q1, t2, b2, q2 = _both(*e, rr_base=0)
    assert np.array_equal(q1, q2)


def test_noalloc_route_rejects_batches_beyond_its_scratch():
    from paper_2607_08565_amd import smetric as S
    n_max = S.route_seq_noalloc_max_req()
    assert n_max == 65536
    small = [to_dev(x) for x in _batch(np.random.default_rng(72), 4, 8)]
    tgt = torch.empty(4, dtype=torch.int32, device="cuda")
    br = torch.empty(4, dtype=torch.uint8, device="cuda")
    p = S._Params(**W.DEFAULT_PARAMS)
    # the C call returns before any launch: the size check precedes all GPU work
    rc = S._lib.smetric_route_seq_noalloc(
        C.c_void_p(small[0].data_ptr()), n_max + 1, 8, C.c_void_p(small[1].data_ptr()),
        C.c_void_p(small[2].data_ptr()), C.c_void_p(small[3].data_ptr()), C.c_void_p(small[4].data_ptr()),
        C.byref(p), C.c_uint64(0), C.c_void_p(tgt.data_ptr()), C.c_void_p(br.data_ptr()), None, S._stream())
    assert rc == S.EWORKSPACE
