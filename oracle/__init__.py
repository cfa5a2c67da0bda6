"""SMetric oracle: plain sequential CPU definition of the matching/routing hot path.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg import this package; the product library never does.  The C++ source
(``smetric_oracle.cpp``) shares no code with the GPU library; this module only marshals
numpy arrays into it with ctypes.

Paper: "SMetric: Rethink LLM Scheduling for Serving Agents with Balanced
Session-centric Scheduling" (arXiv 2607.08565).  Which passage each function follows is
stated in the C++ source next to it.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "smetric_oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")
# a separately built copy (e.g. the sanitizer build the tests make) may be named here
_LIB_OVERRIDE = os.environ.get("SMETRIC_ORACLE_LIB")

OK, EINVAL, EFULL = 0, -1, -2
BRANCH_NAMES = {0: "first-turn", 1: "evicted", 2: "stick", 3: "last-resort", 4: "migrate", 5: "migrate-tpot",
                6: "scored", 7: "hit-filter", 255: "invalid"}


def build(extra_flags: tuple[str, ...] = (), out: str | None = None) -> str:
    """Compile the oracle with g++ (always recompiles). Returns the library path."""
    out = out or _LIB
    cmd = ["g++", "-O2", "-std=c++17", "-Wall", "-Wextra", "-shared", "-fPIC", *extra_flags, _SRC, "-o", out]
    subprocess.run(cmd, check=True)
    return out


class _Params(C.Structure):
    _fields_ = [
        ("c_lin", C.c_int64),
        ("c_att", C.c_int64),
        ("slo_b", C.c_int64),
        ("slo_a", C.c_int64),
        ("slack_num", C.c_int32),
        ("slack_den", C.c_int32),
        ("hit_num", C.c_int32),
        ("hit_den", C.c_int32),
        ("block_size", C.c_int32),
    ]


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if _LIB_OVERRIDE:
        lib = C.CDLL(_LIB_OVERRIDE)
    else:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = C.CDLL(_LIB)
    P = C.c_void_p
    lib.orc_hash_blocks.argtypes = [P, P, C.c_int32, C.c_int32, C.c_uint64, P, P]
    lib.orc_hash_consts.argtypes = [C.c_uint64, C.c_int32, P, P, P]
    lib.orc_splitmix_next.argtypes = [P]
    lib.orc_splitmix_next.restype = C.c_uint64
    lib.orc_index_new.argtypes = [C.c_uint64, C.c_int32]
    lib.orc_index_new.restype = C.c_void_p
    lib.orc_index_free.argtypes = [P]
    lib.orc_index_size.argtypes = [P]
    lib.orc_index_size.restype = C.c_uint64
    lib.orc_index_status.argtypes = [P]
    lib.orc_index_insert.argtypes = [P, P, P, C.c_int32, C.c_int64, P, P, C.c_uint32]
    lib.orc_index_evict.argtypes = [P, C.c_uint32, C.c_uint32]
    lib.orc_index_dump.argtypes = [P, P, P, C.c_uint64]
    lib.orc_index_dump.restype = C.c_uint64
    lib.orc_match.argtypes = [P, P, P, C.c_int32, C.c_int64, P]
    lib.orc_route.argtypes = [P, C.c_int32, C.c_int32, P, P, P, P, C.POINTER(_Params), C.c_uint64, P, P]
    lib.orc_route_loadaware.argtypes = [P, C.c_int32, C.c_int32, P, P, P, P, P, C.c_int32, C.c_int32,
                                        C.POINTER(_Params), C.c_uint64, P, P]
    lib.orc_imbalance.argtypes = [P, P, P, C.c_int64, C.c_int32, C.c_int64, C.c_int32, P, P, P]
    lib.orc_sessions.argtypes = [P, P, C.c_int32, C.c_int64, P, P, P, P]
    lib.orc_route_seq.argtypes = [P, C.c_int32, C.c_int32, P, P, P, P, C.POINTER(_Params), C.c_uint64, P, P, P]
    lib.orc_route_coloc.argtypes = [P, C.c_int32, C.c_int32, P, P, P, P, P, P, C.POINTER(_Params), C.c_uint64,
                                    P, P]
    lib.orc_test_prod_less.argtypes = [C.c_int64, C.c_uint64, C.c_uint64, C.c_int64, C.c_uint64, C.c_uint64]
    lib.orc_route_seq_coloc.argtypes = [P, C.c_int32, C.c_int32, P, P, P, P, P, P, C.POINTER(_Params), C.c_uint64,
                                        P, P, P, P]
    lib.orc_route_score.argtypes = [C.c_int32, P, C.c_int32, C.c_int32, P, P, P, C.c_int32, C.c_int32, C.c_int32,
                                    C.c_uint64, P, P]
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(C.c_void_p)


def _arr(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def splitmix_stream(seed: int, n: int) -> list[int]:
    st = C.c_uint64(seed)
    lib = _load()
    return [int(lib.orc_splitmix_next(C.byref(st))) for _ in range(n)]


def hash_consts(seed: int, block_size: int = 16):
    K = np.zeros(block_size, np.uint32)
    M = C.c_uint64()
    s0 = C.c_uint64()
    rc = _load().orc_hash_consts(C.c_uint64(seed), block_size, _ptr(K), C.byref(M), C.byref(s0))
    if rc != OK:
        raise ValueError(f"orc_hash_consts rc={rc}")
    return K, int(M.value), int(s0.value)


def hash_blocks(tokens, tok_off, block_size: int = 16, seed: int = 0):
    """Returns (blk_off int64[R+1], keys uint64[N_blk])."""
    tokens = _arr(tokens, np.int32)
    tok_off = _arr(tok_off, np.int64)
    R = len(tok_off) - 1
    lens = np.diff(tok_off)
    n_blk = int((lens // block_size).sum()) if R > 0 else 0
    blk_off = np.zeros(R + 1, np.int64)
    keys = np.zeros(max(n_blk, 1), np.uint64)
    rc = _load().orc_hash_blocks(_ptr(tokens) if len(tokens) else None, _ptr(tok_off), R, block_size,
                                 C.c_uint64(seed), _ptr(blk_off), _ptr(keys))
    if rc != OK:
        raise ValueError(f"orc_hash_blocks rc={rc}")
    return blk_off, keys[:n_blk]


class Index:
    """The oracle's block index: a set of (key, instance) entries with session/epoch."""

    def __init__(self, capacity: int, n_instances: int):
        self._lib = _load()
        self.n_instances = n_instances
        self._h = self._lib.orc_index_new(C.c_uint64(capacity), n_instances)
        if not self._h:
            raise ValueError("bad index parameters")

    def __del__(self):
        if getattr(self, "_h", None):
            self._lib.orc_index_free(self._h)
            self._h = None

    @property
    def size(self) -> int:
        return int(self._lib.orc_index_size(self._h))

    @property
    def status(self) -> int:
        return int(self._lib.orc_index_status(self._h))

    def insert(self, keys, blk_off, instance, session, epoch: int, n_blocks: int | None = None) -> int:
        keys = _arr(keys, np.uint64)
        blk_off = _arr(blk_off, np.int64)
        R = len(blk_off) - 1
        instance = _arr(instance, np.int32)
        session = _arr(session, np.uint32)
        nb = len(keys) if n_blocks is None else n_blocks
        kbuf = keys if len(keys) else np.zeros(1, np.uint64)
        return int(self._lib.orc_index_insert(self._h, _ptr(kbuf), _ptr(blk_off), R, C.c_int64(nb),
                                              _ptr(instance) if R else None, _ptr(session) if R else None,
                                              C.c_uint32(epoch)))

    def evict(self, num: int, den: int) -> int:
        return int(self._lib.orc_index_evict(self._h, C.c_uint32(num), C.c_uint32(den)))

    def dump(self):
        n = self.size
        keys = np.zeros(max(n, 1), np.uint64)
        vals = np.zeros(max(n, 1), np.uint64)
        got = int(self._lib.orc_index_dump(self._h, _ptr(keys), _ptr(vals), C.c_uint64(n)))
        assert got == n
        return keys[:n], vals[:n]

    def match(self, keys, blk_off, n_blocks: int | None = None) -> np.ndarray:
        keys = _arr(keys, np.uint64)
        blk_off = _arr(blk_off, np.int64)
        R = len(blk_off) - 1
        out = np.zeros((max(R, 0), self.n_instances), np.int32)
        nb = len(keys) if n_blocks is None else n_blocks
        kbuf = keys if len(keys) else np.zeros(1, np.uint64)
        self.last_rc = int(self._lib.orc_match(self._h, _ptr(kbuf), _ptr(blk_off), R, C.c_int64(nb),
                                               _ptr(out) if out.size else None))
        return out


def unpack_vals(vals: np.ndarray):
    """Dump value layout: instance << 48 | epoch << 24 | session."""
    vals = np.asarray(vals, np.uint64)
    inst = (vals >> np.uint64(48)).astype(np.int64)
    epoch = ((vals >> np.uint64(24)) & np.uint64(0xFFFFFF)).astype(np.int64)
    sess = (vals & np.uint64(0xFFFFFF)).astype(np.int64)
    return inst, epoch, sess


def route(matched, prompt_len, hist_len, turn, q, params: dict, rr_base: int = 0):
    """Returns (target int32[R], branch uint8[R]); raises on invalid parameters."""
    matched = _arr(matched, np.int32)
    R, I = matched.shape
    prompt_len = _arr(prompt_len, np.int32)
    hist_len = _arr(hist_len, np.int32)
    turn = _arr(turn, np.int32)
    q = _arr(q, np.int64)
    p = _Params(**params)
    target = np.zeros(max(R, 1), np.int32)
    branch = np.zeros(max(R, 1), np.uint8)
    rc = _load().orc_route(_ptr(matched) if matched.size else None, R, I,
                           _ptr(prompt_len) if R else None, _ptr(hist_len) if R else None,
                           _ptr(turn) if R else None, _ptr(q), C.byref(p), C.c_uint64(rr_base),
                           _ptr(target), _ptr(branch))
    if rc != OK:
        raise ValueError(f"orc_route rc={rc}")
    return target[:R], branch[:R]


# Per-instance decode slack at or above this value means "no live decode" (App. B's
# all() over an empty set is true).
NO_DECODE = 1 << 62


def route_coloc(matched, prompt_len, hist_len, turn, q, slack, n_run, params: dict, rr_base: int = 0):
    """The rule under PD colocation (App. B pseudocode). slack: int64[I] smallest slack of the
    instance's live decodes in ns (>= NO_DECODE: none); n_run: int32[I] requests at the
    instance. Returns (target int32[R], branch uint8[R]); raises on invalid parameters."""
    matched = _arr(matched, np.int32)
    R, I = matched.shape
    prompt_len = _arr(prompt_len, np.int32)
    hist_len = _arr(hist_len, np.int32)
    turn = _arr(turn, np.int32)
    q = _arr(q, np.int64)
    slack = _arr(slack, np.int64)
    n_run = _arr(n_run, np.int32)
    p = _Params(**params)
    target = np.zeros(max(R, 1), np.int32)
    branch = np.zeros(max(R, 1), np.uint8)
    rc = _load().orc_route_coloc(_ptr(matched) if matched.size else None, R, I,
                                 _ptr(prompt_len) if R else None, _ptr(hist_len) if R else None,
                                 _ptr(turn) if R else None, _ptr(q), _ptr(slack), _ptr(n_run), C.byref(p),
                                 C.c_uint64(rr_base), _ptr(target), _ptr(branch))
    if rc != OK:
        raise ValueError(f"orc_route_coloc rc={rc}")
    return target[:R], branch[:R]


def route_seq(matched, prompt_len, hist_len, turn, q, params: dict, rr_base: int = 0):
    """Requests routed one at a time, each seeing the queue updated by the earlier ones.
    Returns (target int32[R], branch uint8[R], q_after int64[I] in ns, rounded down)."""
    matched = _arr(matched, np.int32)
    R, I = matched.shape
    prompt_len = _arr(prompt_len, np.int32)
    hist_len = _arr(hist_len, np.int32)
    turn = _arr(turn, np.int32)
    q = _arr(q, np.int64)
    p = _Params(**params)
    target = np.zeros(max(R, 1), np.int32)
    branch = np.zeros(max(R, 1), np.uint8)
    q_out = np.zeros(I, np.int64)
    rc = _load().orc_route_seq(_ptr(matched) if matched.size else None, R, I,
                               _ptr(prompt_len) if R else None, _ptr(hist_len) if R else None,
                               _ptr(turn) if R else None, _ptr(q), C.byref(p), C.c_uint64(rr_base),
                               _ptr(target), _ptr(branch), _ptr(q_out))
    if rc != OK:
        raise ValueError(f"orc_route_seq rc={rc}")
    return target[:R], branch[:R], q_out


def route_seq_coloc(matched, prompt_len, hist_len, turn, q, slack, n_run, params: dict, rr_base: int = 0):
    """The rule under PD colocation with requests taken one at a time: each decided by
    route_coloc on the state the earlier ones left (their prefill queued on their target,
    one more request there).  Returns (target int32[R], branch uint8[R], q_after int64[I]
    in ns rounded down, n_after int64[I])."""
    matched = _arr(matched, np.int32)
    R, I = matched.shape
    prompt_len = _arr(prompt_len, np.int32)
    hist_len = _arr(hist_len, np.int32)
    turn = _arr(turn, np.int32)
    q = _arr(q, np.int64)
    slack = _arr(slack, np.int64)
    n_run = _arr(n_run, np.int32)
    p = _Params(**params)
    target = np.zeros(max(R, 1), np.int32)
    branch = np.zeros(max(R, 1), np.uint8)
    q_out = np.zeros(I, np.int64)
    n_out = np.zeros(I, np.int64)
    rc = _load().orc_route_seq_coloc(_ptr(matched) if matched.size else None, R, I,
                                     _ptr(prompt_len) if R else None, _ptr(hist_len) if R else None,
                                     _ptr(turn) if R else None, _ptr(q), _ptr(slack), _ptr(n_run), C.byref(p),
                                     C.c_uint64(rr_base), _ptr(target), _ptr(branch), _ptr(q_out), _ptr(n_out))
    if rc != OK:
        raise ValueError(f"orc_route_seq_coloc rc={rc}")
    return target[:R], branch[:R], q_out, n_out


def test_prod_less(a: int, x: int, b: int, y: int) -> bool:
    """The oracle's exact a * x < b * y (0 <= a, b < 2^127; 0 <= x, y < 2^64)."""
    m = (1 << 64) - 1
    return bool(_load().orc_test_prod_less(a >> 64, a & m, x, b >> 64, b & m, y))


def sessions(keys, blk_off, user, turn):
    """App. A session reconstruction.  Returns (parent int32[R], session int32[R])."""
    keys = _arr(keys, np.uint64)
    blk_off = _arr(blk_off, np.int64)
    user = _arr(user, np.uint32)
    turn = _arr(turn, np.int32)
    R = len(blk_off) - 1
    parent = np.zeros(max(R, 1), np.int32)
    session = np.zeros(max(R, 1), np.int32)
    rc = _load().orc_sessions(_ptr(keys) if len(keys) else None, _ptr(blk_off), R, int(len(keys)),
                              _ptr(user) if R else None, _ptr(turn) if R else None, _ptr(parent), _ptr(session))
    if rc != OK:
        raise ValueError(f"orc_sessions rc={rc}")
    return parent[:R], session[:R]


def route_loadaware(matched, prompt_len, hist_len, turn, q, load, margin: tuple[int, int], params: dict,
                    rr_base: int = 0):
    """Sec. 5.4 ablation: session stickiness with the load-aware filter (leave prev when its load
    exceeds the mean by margin = num/den; den 0 = never).  Returns (target, branch)."""
    matched = _arr(matched, np.int32)
    R, I = matched.shape
    prompt_len, hist_len, turn = _arr(prompt_len, np.int32), _arr(hist_len, np.int32), _arr(turn, np.int32)
    q, load = _arr(q, np.int64), _arr(load, np.int64)
    p = _Params(**params)
    target = np.zeros(max(R, 1), np.int32)
    branch = np.zeros(max(R, 1), np.uint8)
    rc = _load().orc_route_loadaware(_ptr(matched) if matched.size else None, R, I,
                                     _ptr(prompt_len) if R else None, _ptr(hist_len) if R else None,
                                     _ptr(turn) if R else None, _ptr(q), _ptr(load), int(margin[0]), int(margin[1]),
                                     C.byref(p), C.c_uint64(rr_base), _ptr(target), _ptr(branch))
    if rc != OK:
        raise ValueError(f"orc_route_loadaware rc={rc}")
    return target[:R], branch[:R]


def imbalance(inst, t0, t1, n_inst: int, window: int, n_windows: int):
    """Per-window (sum, max) of instance loads (running requests x window length).
    Returns (sum int64[W], max int64[W], n_bad)."""
    inst, t0, t1 = _arr(inst, np.int32), _arr(t0, np.int64), _arr(t1, np.int64)
    out_sum = np.zeros(max(n_windows, 1), np.int64)
    out_max = np.zeros(max(n_windows, 1), np.int64)
    bad = C.c_int64(0)
    rc = _load().orc_imbalance(_ptr(inst) if len(inst) else None, _ptr(t0) if len(t0) else None,
                               _ptr(t1) if len(t1) else None, len(inst), n_inst, window, n_windows,
                               _ptr(out_sum), _ptr(out_max), C.byref(bad))
    if rc != OK:
        raise ValueError(f"orc_imbalance rc={rc}")
    return out_sum[:n_windows], out_max[:n_windows], bad.value


SCORE_LOAD, SCORE_TOKENS, SCORE_PRODUCT, SCORE_LINEAR, SCORE_HIT_FILTER = range(5)


def route_score(kind, matched, prompt_len, q, load, block_size, lam=(0, 1), rr_base: int = 0):
    """The scoring template's comparison scorers (Sec. 4.1, Sec. 5): argmin over instances of
    f(kind), ties in rotation order. q: int64[I] queued prefill tokens; load: int32[I] batch
    sizes; lam = (num, den) for the weighted sum (kinds 3 and 4). Returns (target int32[R],
    branch uint8[R]: 6 scored, 7 hit filter, 255 out of domain); raises on bad scalars."""
    matched = _arr(matched, np.int32)
    R, I = matched.shape
    prompt_len = _arr(prompt_len, np.int32)
    q = _arr(q, np.int64)
    load = _arr(load, np.int32)
    target = np.zeros(max(R, 1), np.int32)
    branch = np.zeros(max(R, 1), np.uint8)
    rc = _load().orc_route_score(int(kind), _ptr(matched) if matched.size else None, R, I,
                                 _ptr(prompt_len) if R else None, _ptr(q), _ptr(load), int(block_size),
                                 int(lam[0]), int(lam[1]), C.c_uint64(rr_base), _ptr(target), _ptr(branch))
    if rc != OK:
        raise ValueError(f"orc_route_score rc={rc}")
    return target[:R], branch[:R]
