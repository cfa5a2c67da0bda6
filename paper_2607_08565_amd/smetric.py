"""Thin ctypes binding of libsmetric.so (C ABI in include/smetric.h).

Argument marshalling only: device tensors are passed by data pointer, the stream is
torch's current stream, and every step runs in the library's HIP kernels.  Importing
this module loads the library and raises if it has not been built -- there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

from .workload import BLOCK, DEFAULT_SEED

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsmetric.so")

OK, EINVAL, EFULL, EHIP, EWORKSPACE, EINTERNAL = 0, -1, -2, -3, -4, -5
FIRST_TURN, EVICTED, STICK, LAST_RESORT, MIGRATE, INVALID = 0, 1, 2, 3, 4, 255


class SmetricError(RuntimeError):
    def __init__(self, fn: str, rc: int):
        super().__init__(f"{fn} returned {rc}")
        self.rc = rc


class _Index(C.Structure):
    _fields_ = [
        ("mem", C.c_void_p), ("mem_bytes", C.c_uint64), ("capacity", C.c_uint64),
        ("n_instances", C.c_int32), ("bitmap_words", C.c_int32), ("spill_threshold", C.c_int32),
        ("reserved0", C.c_int32), ("n_buckets", C.c_uint64), ("n_records", C.c_uint64),
        ("slots", C.c_void_p), ("pool", C.c_void_p), ("hdr", C.c_void_p),
    ]


class _Params(C.Structure):
    _fields_ = [
        ("c_lin", C.c_int64), ("c_att", C.c_int64), ("slo_b", C.c_int64), ("slo_a", C.c_int64),
        ("slack_num", C.c_int32), ("slack_den", C.c_int32), ("hit_num", C.c_int32),
        ("hit_den", C.c_int32), ("block_size", C.c_int32),
    ]


def _load() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build the HIP library first (__graft_entry__.build())")
    lib = C.CDLL(LIB_PATH)
    P, I32, I64, U64, U32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_uint32
    PIX = C.POINTER(_Index)
    sig = {
        "smetric_version": [],
        "smetric_block_offsets": [P, I32, I32, P, P],
        "smetric_hash_blocks": [P, I64, P, P, I32, I64, I32, U64, P, P, P],
        "smetric_index_bytes": [U64, I32, U64, P],
        "smetric_index_init": [PIX, P, U64, U64, I32, U64, P],
        "smetric_index_attach": [PIX, P, U64, U64, I32, U64],
        "smetric_index_stats": [PIX, P, P, I32, P],
        "smetric_match": [PIX, P, P, I32, I64, P, P],
        "smetric_route": [P, I32, I32, P, P, P, P, C.POINTER(_Params), U64, P, P, P],
        "smetric_route_coloc": [P, I32, I32, P, P, P, P, P, P, C.POINTER(_Params), U64, P, P, P],
        "smetric_route_seq_ws_bytes": [I32, P],
        "smetric_route_seq_coloc_ws_bytes": [I32, I32, P],
        "smetric_route_loadaware": [P, I32, I32, P, P, P, P, P, I32, I32, C.POINTER(_Params), U64, P, P, P],
        "smetric_imbalance_ws_bytes": [I32, I32, P],
        "smetric_imbalance": [P, P, P, I64, I32, I64, I32, P, P, P, P, U64, P],
        "smetric_sessions_ws_bytes": [I32, P],
        "smetric_sessions": [P, P, I32, I64, P, P, P, P, P, P, U64, P],
        "smetric_route_seq": [P, I32, I32, P, P, P, P, C.POINTER(_Params), U64, P, P, P, P, U64, P],
        "smetric_route_seq_noalloc_max_req": [],
        "smetric_route_seq_noalloc": [P, I32, I32, P, P, P, P, C.POINTER(_Params), U64, P, P, P, P],
        "smetric_route_seq_coloc": [P, I32, I32, P, P, P, P, P, P, C.POINTER(_Params), U64, P, P, P, P, P, U64, P],
        "smetric_index_insert_ws_bytes": [I64, P],
        "smetric_index_insert": [PIX, P, P, I32, I64, P, P, U32, P, U64, P],
        "smetric_index_evict_ws_bytes": [PIX, P],
        "smetric_index_evict": [PIX, U32, U32, P, U64, P],
        "smetric_index_dump": [PIX, P, P, U64, P, U64, P, P],
        "smetric_probe_ws_bytes": [I64, P],
        "smetric_probe": [PIX, P, P, I32, I64, P, U64, P],
        "smetric_probe_partition": [PIX, P, P, I32, I64, P, U64, P],
        "smetric_probe_lookup": [PIX, P, U64, P, P, I32, I64, P],
        "smetric_probe_stats": [P, U64, I64, P, P, P],
        "smetric_hash_partition": [P, I64, P, P, I32, I64, I32, U64, P, P, PIX, P, U64, P],
        "smetric_match_probed": [PIX, P, U64, P, P, I32, I64, P, P],
        "smetric_index_insert_probed": [PIX, P, U64, I32, I64, P, P, U32, P, U64, P],
        "smetric_route_score": [I32, P, I32, I32, P, P, P, I32, I32, I32, U64, P, P, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = C.c_int
    return lib


_lib = _load()
EXPORTED = (
    "smetric_version", "smetric_block_offsets", "smetric_hash_blocks", "smetric_index_bytes",
    "smetric_index_init", "smetric_index_attach", "smetric_index_stats", "smetric_match",
    "smetric_route", "smetric_index_insert_ws_bytes", "smetric_index_insert",
    "smetric_index_evict_ws_bytes", "smetric_index_evict", "smetric_index_dump",
    "smetric_probe_ws_bytes", "smetric_probe", "smetric_match_probed", "smetric_index_insert_probed",
    "smetric_route_coloc", "smetric_route_seq_ws_bytes", "smetric_route_seq", "smetric_sessions_ws_bytes",
    "smetric_sessions", "smetric_route_loadaware", "smetric_imbalance_ws_bytes", "smetric_imbalance",
    "smetric_probe_partition", "smetric_probe_lookup", "smetric_hash_partition", "smetric_route_seq_coloc",
    "smetric_route_seq_coloc_ws_bytes", "smetric_route_seq_noalloc", "smetric_route_seq_noalloc_max_req",
    "smetric_probe_stats", "smetric_route_score",
)


def _check(fn: str, rc: int):
    if rc != OK:
        raise SmetricError(fn, rc)


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t: torch.Tensor, dtype: torch.dtype, name: str) -> C.c_void_p:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or t.dtype != dtype or not t.is_contiguous():
        raise TypeError(f"{name}: expected a contiguous {dtype} CUDA tensor")
    return C.c_void_p(t.data_ptr())


def version() -> int:
    return _lib.smetric_version()


def block_offsets(tok_off, block_size: int = BLOCK):
    """Host helper: (blk_off int64[R+1] numpy, n_blocks)."""
    tok_off = np.ascontiguousarray(np.asarray(tok_off, np.int64))
    R = len(tok_off) - 1
    blk_off = np.zeros(R + 1, np.int64)
    nb = C.c_int64()
    _check("smetric_block_offsets", _lib.smetric_block_offsets(
        tok_off.ctypes.data_as(C.c_void_p), R, block_size, blk_off.ctypes.data_as(C.c_void_p), C.byref(nb)))
    return blk_off, int(nb.value)


def hash_blocks(tokens: torch.Tensor, tok_off: torch.Tensor, blk_off: torch.Tensor, n_blocks: int,
                block_size: int = BLOCK, seed: int = DEFAULT_SEED, keys: torch.Tensor | None = None,
                status: torch.Tensor | None = None) -> torch.Tensor:
    R = tok_off.numel() - 1
    if keys is None:
        keys = torch.empty(max(n_blocks, 1), dtype=torch.uint64, device=tokens.device)
    _check("smetric_hash_blocks", _lib.smetric_hash_blocks(
        _dev(tokens, torch.int32, "tokens"), tokens.numel(), _dev(tok_off, torch.int64, "tok_off"),
        _dev(blk_off, torch.int64, "blk_off"), R, n_blocks, block_size, C.c_uint64(seed),
        _dev(keys, torch.uint64, "keys"), _dev(status, torch.int32, "status") if status is not None else None,
        _stream()))
    return keys


def route(matched: torch.Tensor, prompt_len: torch.Tensor, hist_len: torch.Tensor, turn: torch.Tensor,
          q: torch.Tensor, params: dict, rr_base: int = 0, target: torch.Tensor | None = None,
          branch: torch.Tensor | None = None):
    R, I = matched.shape
    dev = matched.device
    target = torch.empty(max(R, 1), dtype=torch.int32, device=dev) if target is None else target
    branch = torch.empty(max(R, 1), dtype=torch.uint8, device=dev) if branch is None else branch
    p = _Params(**params)
    _check("smetric_route", _lib.smetric_route(
        _dev(matched, torch.int32, "matched"), R, I, _dev(prompt_len, torch.int32, "prompt_len"),
        _dev(hist_len, torch.int32, "hist_len"), _dev(turn, torch.int32, "turn"), _dev(q, torch.int64, "q"),
        C.byref(p), C.c_uint64(rr_base), _dev(target, torch.int32, "target"), _dev(branch, torch.uint8, "branch"),
        _stream()))
    return target[:R], branch[:R]



def route_seq_ws_bytes(n_req: int) -> int:
    b = C.c_uint64(0)
    _check("smetric_route_seq_ws_bytes", _lib.smetric_route_seq_ws_bytes(n_req, C.byref(b)))
    return b.value


def route_seq_coloc_ws_bytes(n_req: int, n_instances: int) -> int:
    b = C.c_uint64(0)
    _check("smetric_route_seq_coloc_ws_bytes", _lib.smetric_route_seq_coloc_ws_bytes(n_req, n_instances, C.byref(b)))
    return b.value


def route_seq(matched: torch.Tensor, prompt_len: torch.Tensor, hist_len: torch.Tensor, turn: torch.Tensor,
              q: torch.Tensor, params: dict, rr_base: int = 0, target: torch.Tensor | None = None,
              branch: torch.Tensor | None = None, q_out: torch.Tensor | None = None,
              workspace: torch.Tensor | None = None):
    """smetric_route_seq: requests routed one at a time, each seeing the earlier ones' load.
    Returns (target, branch, q_out)."""
    R, I = matched.shape
    dev = matched.device
    target = torch.empty(max(R, 1), dtype=torch.int32, device=dev) if target is None else target
    branch = torch.empty(max(R, 1), dtype=torch.uint8, device=dev) if branch is None else branch
    q_out = torch.empty(I, dtype=torch.int64, device=dev) if q_out is None else q_out
    need = route_seq_ws_bytes(R)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    p = _Params(**params)
    _check("smetric_route_seq", _lib.smetric_route_seq(
        _dev(matched, torch.int32, "matched"), R, I, _dev(prompt_len, torch.int32, "prompt_len"),
        _dev(hist_len, torch.int32, "hist_len"), _dev(turn, torch.int32, "turn"), _dev(q, torch.int64, "q"),
        C.byref(p), C.c_uint64(rr_base), _dev(target, torch.int32, "target"), _dev(branch, torch.uint8, "branch"),
        _dev(q_out, torch.int64, "q_out"), _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream()))
    return target[:R], branch[:R], q_out

def route_seq_noalloc(matched: torch.Tensor, prompt_len: torch.Tensor, hist_len: torch.Tensor, turn: torch.Tensor,
                      q: torch.Tensor, params: dict, rr_base: int, target: torch.Tensor, branch: torch.Tensor,
                      q_out: torch.Tensor | None = None):
    """smetric_route_seq_noalloc: smetric_route_seq with the library's own scratch (no
    workspace; at most route_seq_noalloc_max_req() requests).  The caller supplies the
    outputs, so the call allocates nothing.  Returns (target, branch, q_out)."""
    R, I = matched.shape
    if R > route_seq_noalloc_max_req():
        raise SmetricError("smetric_route_seq_noalloc", EWORKSPACE)
    p = _Params(**params)
    _check("smetric_route_seq_noalloc", _lib.smetric_route_seq_noalloc(
        _dev(matched, torch.int32, "matched"), R, I, _dev(prompt_len, torch.int32, "prompt_len"),
        _dev(hist_len, torch.int32, "hist_len"), _dev(turn, torch.int32, "turn"), _dev(q, torch.int64, "q"),
        C.byref(p), C.c_uint64(rr_base), _dev(target, torch.int32, "target"), _dev(branch, torch.uint8, "branch"),
        None if q_out is None else _dev(q_out, torch.int64, "q_out"), _stream()))
    return target[:R], branch[:R], q_out


def route_seq_noalloc_max_req() -> int:
    return int(_lib.smetric_route_seq_noalloc_max_req())


def route_seq_coloc(matched: torch.Tensor, prompt_len: torch.Tensor, hist_len: torch.Tensor, turn: torch.Tensor,
                    q: torch.Tensor, tpot_slack: torch.Tensor, n_running: torch.Tensor, params: dict,
                    rr_base: int = 0, target: torch.Tensor | None = None, branch: torch.Tensor | None = None,
                    q_out: torch.Tensor | None = None, n_out: torch.Tensor | None = None,
                    workspace: torch.Tensor | None = None):
    """smetric_route_seq_coloc: the colocation rule with requests routed one at a time.
    Returns (target, branch, q_out, n_out)."""
    R, I = matched.shape
    dev = matched.device
    target = torch.empty(max(R, 1), dtype=torch.int32, device=dev) if target is None else target
    branch = torch.empty(max(R, 1), dtype=torch.uint8, device=dev) if branch is None else branch
    q_out = torch.empty(I, dtype=torch.int64, device=dev) if q_out is None else q_out
    n_out = torch.empty(I, dtype=torch.int64, device=dev) if n_out is None else n_out
    need = route_seq_coloc_ws_bytes(R, I) if 1 <= I <= 4096 else 256  # else the call reports EINVAL
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    p = _Params(**params)
    _check("smetric_route_seq_coloc", _lib.smetric_route_seq_coloc(
        _dev(matched, torch.int32, "matched"), R, I, _dev(prompt_len, torch.int32, "prompt_len"),
        _dev(hist_len, torch.int32, "hist_len"), _dev(turn, torch.int32, "turn"), _dev(q, torch.int64, "q"),
        _dev(tpot_slack, torch.int64, "tpot_slack"), _dev(n_running, torch.int32, "n_running"), C.byref(p),
        C.c_uint64(rr_base), _dev(target, torch.int32, "target"), _dev(branch, torch.uint8, "branch"),
        _dev(q_out, torch.int64, "q_out"), _dev(n_out, torch.int64, "n_out"),
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream()))
    return target[:R], branch[:R], q_out, n_out


def route_loadaware(matched: torch.Tensor, prompt_len: torch.Tensor, hist_len: torch.Tensor, turn: torch.Tensor,
                    q: torch.Tensor, load: torch.Tensor, margin: tuple[int, int], params: dict, rr_base: int = 0,
                    target: torch.Tensor | None = None, branch: torch.Tensor | None = None):
    """smetric_route_loadaware: the Sec. 5.4 ablation's load-aware filter."""
    R, I = matched.shape
    dev = matched.device
    target = torch.empty(max(R, 1), dtype=torch.int32, device=dev) if target is None else target
    branch = torch.empty(max(R, 1), dtype=torch.uint8, device=dev) if branch is None else branch
    p = _Params(**params)
    _check("smetric_route_loadaware", _lib.smetric_route_loadaware(
        _dev(matched, torch.int32, "matched"), R, I, _dev(prompt_len, torch.int32, "prompt_len"),
        _dev(hist_len, torch.int32, "hist_len"), _dev(turn, torch.int32, "turn"), _dev(q, torch.int64, "q"),
        _dev(load, torch.int64, "load"), int(margin[0]), int(margin[1]), C.byref(p), C.c_uint64(rr_base),
        _dev(target, torch.int32, "target"), _dev(branch, torch.uint8, "branch"), _stream()))
    return target[:R], branch[:R]


def imbalance(inst: torch.Tensor, t0: torch.Tensor, t1: torch.Tensor, n_inst: int, window: int, n_windows: int,
              workspace: torch.Tensor | None = None):
    """smetric_imbalance: per-window (sum, max) of instance loads.  Returns (sum, max, n_bad)."""
    dev = inst.device
    b = C.c_uint64(0)
    _check("smetric_imbalance_ws_bytes", _lib.smetric_imbalance_ws_bytes(n_inst, n_windows, C.byref(b)))
    if workspace is None or workspace.numel() < b.value:
        workspace = torch.empty(b.value, dtype=torch.uint8, device=dev)
    out_sum = torch.empty(max(n_windows, 1), dtype=torch.int64, device=dev)
    out_max = torch.empty(max(n_windows, 1), dtype=torch.int64, device=dev)
    n_bad = torch.empty(1, dtype=torch.int64, device=dev)
    _check("smetric_imbalance", _lib.smetric_imbalance(
        _dev(inst, torch.int32, "inst"), _dev(t0, torch.int64, "t0"), _dev(t1, torch.int64, "t1"), inst.numel(),
        n_inst, window, n_windows, _dev(out_sum, torch.int64, "out_sum"), _dev(out_max, torch.int64, "out_max"),
        _dev(n_bad, torch.int64, "n_bad"), _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream()))
    return out_sum[:n_windows], out_max[:n_windows], n_bad


def sessions_ws_bytes(n_req: int) -> int:
    b = C.c_uint64(0)
    _check("smetric_sessions_ws_bytes", _lib.smetric_sessions_ws_bytes(n_req, C.byref(b)))
    return b.value


def sessions(keys: torch.Tensor, blk_off: torch.Tensor, n_blocks: int, user: torch.Tensor, turn: torch.Tensor,
             parent: torch.Tensor | None = None, session: torch.Tensor | None = None,
             status: torch.Tensor | None = None, workspace: torch.Tensor | None = None):
    """smetric_sessions: App. A session reconstruction.  Returns (parent, session)."""
    R = blk_off.numel() - 1
    dev = blk_off.device
    parent = torch.empty(max(R, 1), dtype=torch.int32, device=dev) if parent is None else parent
    session = torch.empty(max(R, 1), dtype=torch.int32, device=dev) if session is None else session
    need = sessions_ws_bytes(R)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    _check("smetric_sessions", _lib.smetric_sessions(
        _dev(keys, torch.uint64, "keys"), _dev(blk_off, torch.int64, "blk_off"), R, n_blocks,
        _dev(user, torch.uint32, "user"), _dev(turn, torch.int32, "turn"), _dev(parent, torch.int32, "parent"),
        _dev(session, torch.int32, "session"), _dev(status, torch.int32, "status") if status is not None else None,
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream()))
    return parent[:R], session[:R]

# Decode slack at or above this value means "no live decode" (smetric_route_coloc).
NO_DECODE = 1 << 62


def route_coloc(matched: torch.Tensor, prompt_len: torch.Tensor, hist_len: torch.Tensor, turn: torch.Tensor,
                q: torch.Tensor, tpot_slack: torch.Tensor, n_running: torch.Tensor, params: dict, rr_base: int = 0,
                target: torch.Tensor | None = None, branch: torch.Tensor | None = None):
    """smetric_route_coloc: the decision under PD colocation (App. B)."""
    R, I = matched.shape
    dev = matched.device
    target = torch.empty(max(R, 1), dtype=torch.int32, device=dev) if target is None else target
    branch = torch.empty(max(R, 1), dtype=torch.uint8, device=dev) if branch is None else branch
    p = _Params(**params)
    _check("smetric_route_coloc", _lib.smetric_route_coloc(
        _dev(matched, torch.int32, "matched"), R, I, _dev(prompt_len, torch.int32, "prompt_len"),
        _dev(hist_len, torch.int32, "hist_len"), _dev(turn, torch.int32, "turn"), _dev(q, torch.int64, "q"),
        _dev(tpot_slack, torch.int64, "tpot_slack"), _dev(n_running, torch.int32, "n_running"),
        C.byref(p), C.c_uint64(rr_base), _dev(target, torch.int32, "target"), _dev(branch, torch.uint8, "branch"),
        _stream()))
    return target[:R], branch[:R]

# Scorer kinds of smetric_route_score (Sec. 4.1 scoring template).
SCORE_LOAD, SCORE_TOKENS, SCORE_PRODUCT, SCORE_LINEAR, SCORE_HIT_FILTER = range(5)


def route_score(kind: int, matched: torch.Tensor, prompt_len: torch.Tensor, q: torch.Tensor, load: torch.Tensor,
                block_size: int, lam: tuple[int, int] = (0, 1), rr_base: int = 0,
                target: torch.Tensor | None = None, branch: torch.Tensor | None = None):
    """smetric_route_score: argmin of a comparison scorer (q in tokens, load int32 batch
    sizes, lam = (num, den) for the weighted sum and the hit filter)."""
    R, I = matched.shape
    dev = matched.device
    target = torch.empty(max(R, 1), dtype=torch.int32, device=dev) if target is None else target
    branch = torch.empty(max(R, 1), dtype=torch.uint8, device=dev) if branch is None else branch
    _check("smetric_route_score", _lib.smetric_route_score(
        int(kind), _dev(matched, torch.int32, "matched"), R, I, _dev(prompt_len, torch.int32, "prompt_len"),
        _dev(q, torch.int64, "q"), _dev(load, torch.int32, "load"), int(block_size), int(lam[0]), int(lam[1]),
        C.c_uint64(rr_base), _dev(target, torch.int32, "target"), _dev(branch, torch.uint8, "branch"), _stream()))
    return target[:R], branch[:R]


def insert_ws_bytes(n_blocks: int) -> int:
    b = C.c_uint64()
    _check("smetric_index_insert_ws_bytes", _lib.smetric_index_insert_ws_bytes(n_blocks, C.byref(b)))
    return int(b.value)


def probe_ws_bytes(n_blocks: int) -> int:
    b = C.c_uint64()
    _check("smetric_probe_ws_bytes", _lib.smetric_probe_ws_bytes(n_blocks, C.byref(b)))
    return int(b.value)


def index_bytes(capacity: int, n_instances: int, n_slots: int = 0) -> int:
    b = C.c_uint64()
    _check("smetric_index_bytes", _lib.smetric_index_bytes(C.c_uint64(capacity), n_instances, C.c_uint64(n_slots),
                                                           C.byref(b)))
    return int(b.value)


class Index:
    """Global block index in one device buffer (torch-allocated).  n_slots = 0: the
    library's default sizing (at most 3/4 full at capacity); else the table's slot count."""

    def __init__(self, capacity: int, n_instances: int, device="cuda", mem: torch.Tensor | None = None,
                 n_slots: int = 0, _attach: bool = False):
        self.capacity, self.n_instances, self.n_slots_arg = capacity, n_instances, n_slots
        nbytes = index_bytes(capacity, n_instances, n_slots)
        self.mem = torch.empty(nbytes, dtype=torch.uint8, device=device) if mem is None else mem
        self.c = _Index()
        if _attach:
            _check("smetric_index_attach", _lib.smetric_index_attach(
                C.byref(self.c), C.c_void_p(self.mem.data_ptr()), self.mem.numel(), C.c_uint64(capacity),
                n_instances, C.c_uint64(n_slots)))
        else:
            _check("smetric_index_init", _lib.smetric_index_init(
                C.byref(self.c), C.c_void_p(self.mem.data_ptr()), self.mem.numel(), C.c_uint64(capacity),
                n_instances, C.c_uint64(n_slots), _stream()))
        self._ws = None

    @classmethod
    def attach(cls, mem: torch.Tensor, capacity: int, n_instances: int, n_slots: int = 0) -> "Index":
        """An index over `mem`, whose bytes are a copy of an index laid out with the same
        capacity, n_instances and n_slots (smetric_index_attach: nothing is cleared)."""
        return cls(capacity, n_instances, device=mem.device, mem=mem, n_slots=n_slots, _attach=True)

    @property
    def n_slots(self) -> int:
        return int(self.c.n_buckets) * 8

    @property
    def ref(self):
        return C.byref(self.c)

    def _workspace(self, nbytes: int) -> torch.Tensor:
        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = torch.empty(nbytes, dtype=torch.uint8, device=self.mem.device)
        return self._ws

    def stats(self, reset_status: bool = False):
        n, st = C.c_uint64(), C.c_int32()
        _check("smetric_index_stats", _lib.smetric_index_stats(self.ref, C.byref(n), C.byref(st), int(reset_status),
                                                               _stream()))
        return int(n.value), int(st.value)

    def match(self, keys: torch.Tensor, blk_off: torch.Tensor, n_blocks: int,
              matched: torch.Tensor | None = None) -> torch.Tensor:
        R = blk_off.numel() - 1
        if matched is None:
            matched = torch.empty((max(R, 1), self.n_instances), dtype=torch.int32, device=keys.device)
        _check("smetric_match", _lib.smetric_match(
            self.ref, _dev(keys, torch.uint64, "keys"), _dev(blk_off, torch.int64, "blk_off"), R, n_blocks,
            _dev(matched, torch.int32, "matched"), _stream()))
        return matched[:R]

    def insert(self, keys: torch.Tensor, blk_off: torch.Tensor, n_blocks: int, instance: torch.Tensor,
               session: torch.Tensor, epoch: int, workspace: torch.Tensor | None = None):
        R = blk_off.numel() - 1
        need = insert_ws_bytes(n_blocks)
        ws = self._workspace(need) if workspace is None else workspace
        _check("smetric_index_insert", _lib.smetric_index_insert(
            self.ref, _dev(keys, torch.uint64, "keys"), _dev(blk_off, torch.int64, "blk_off"), R, n_blocks,
            _dev(instance, torch.int32, "instance"), _dev(session, torch.int32, "session")
            if session.dtype == torch.int32 else _dev(session, torch.uint32, "session"),
            C.c_uint32(epoch), C.c_void_p(ws.data_ptr()), ws.numel(), _stream()))

    def evict_ws_bytes(self) -> int:
        b = C.c_uint64()
        _check("smetric_index_evict_ws_bytes", _lib.smetric_index_evict_ws_bytes(self.ref, C.byref(b)))
        return int(b.value)

    def evict(self, num: int, den: int):
        ws = self._workspace(self.evict_ws_bytes())
        _check("smetric_index_evict", _lib.smetric_index_evict(self.ref, C.c_uint32(num), C.c_uint32(den),
                                                               C.c_void_p(ws.data_ptr()), ws.numel(), _stream()))

    def dump(self):
        """All entries sorted by (key, instance) as host numpy (keys, vals)."""
        n, _ = self.stats()
        keys = torch.empty(max(n, 1), dtype=torch.uint64, device=self.mem.device)
        vals = torch.empty(max(n, 1), dtype=torch.uint64, device=self.mem.device)
        ws = self._workspace(self.evict_ws_bytes())
        got = C.c_uint64()
        _check("smetric_index_dump", _lib.smetric_index_dump(
            self.ref, C.c_void_p(keys.data_ptr()), C.c_void_p(vals.data_ptr()), C.c_uint64(n),
            C.c_void_p(ws.data_ptr()), ws.numel(), C.byref(got), _stream()))
        assert int(got.value) == n
        return keys[:n].cpu().numpy(), vals[:n].cpu().numpy()

    # region-ordered path: probe once, then match and insert from the probe state
    def probe(self, keys: torch.Tensor, blk_off: torch.Tensor, n_blocks: int, state: torch.Tensor | None = None):
        R = blk_off.numel() - 1
        need = probe_ws_bytes(n_blocks)
        if state is None or state.numel() < need:
            state = torch.empty(need, dtype=torch.uint8, device=keys.device)
        _check("smetric_probe", _lib.smetric_probe(
            self.ref, _dev(keys, torch.uint64, "keys"), _dev(blk_off, torch.int64, "blk_off"), R, n_blocks,
            C.c_void_p(state.data_ptr()), state.numel(), _stream()))
        return state

    def probe_partition(self, keys: torch.Tensor, blk_off: torch.Tensor, n_blocks: int,
                        state: torch.Tensor | None = None):
        """First half of probe(): reads only the index geometry (may overlap an earlier insert)."""
        R = blk_off.numel() - 1
        need = probe_ws_bytes(n_blocks)
        if state is None or state.numel() < need:
            state = torch.empty(need, dtype=torch.uint8, device=keys.device)
        _check("smetric_probe_partition", _lib.smetric_probe_partition(
            self.ref, _dev(keys, torch.uint64, "keys"), _dev(blk_off, torch.int64, "blk_off"), R, n_blocks,
            C.c_void_p(state.data_ptr()), state.numel(), _stream()))
        return state

    def hash_partition(self, tokens: torch.Tensor, tok_off: torch.Tensor, blk_off: torch.Tensor, n_blocks: int,
                       block_size: int = BLOCK, seed: int = DEFAULT_SEED, keys: torch.Tensor | None = None,
                       status: torch.Tensor | None = None, state: torch.Tensor | None = None):
        """hash_blocks + probe_partition in one call; returns (keys, probe state)."""
        R = tok_off.numel() - 1
        if keys is None:
            keys = torch.empty(max(n_blocks, 1), dtype=torch.uint64, device=tokens.device)
        need = probe_ws_bytes(n_blocks)
        if state is None or state.numel() < need:
            state = torch.empty(need, dtype=torch.uint8, device=tokens.device)
        _check("smetric_hash_partition", _lib.smetric_hash_partition(
            _dev(tokens, torch.int32, "tokens"), tokens.numel(), _dev(tok_off, torch.int64, "tok_off"),
            _dev(blk_off, torch.int64, "blk_off"), R, n_blocks, block_size, C.c_uint64(seed),
            _dev(keys, torch.uint64, "keys"), _dev(status, torch.int32, "status") if status is not None else None,
            self.ref, C.c_void_p(state.data_ptr()), state.numel(), _stream()))
        return keys, state

    def probe_lookup(self, state: torch.Tensor, keys: torch.Tensor, blk_off: torch.Tensor, n_blocks: int):
        """Second half of probe(): reads the index (the keys and offsets of the partition)."""
        R = blk_off.numel() - 1
        _check("smetric_probe_lookup", _lib.smetric_probe_lookup(
            self.ref, C.c_void_p(state.data_ptr()), state.numel(), _dev(keys, torch.uint64, "keys"),
            _dev(blk_off, torch.int64, "blk_off"), R, n_blocks, _stream()))
        return state

    @staticmethod
    def probe_stats(state: torch.Tensor, n_blocks: int):
        """(blocks the last lookup on `state` probed, probes of its bound's searches); synchronizes."""
        a, b = C.c_uint64(), C.c_uint64()
        _check("smetric_probe_stats", _lib.smetric_probe_stats(C.c_void_p(state.data_ptr()), state.numel(), n_blocks,
                                                               C.byref(a), C.byref(b), _stream()))
        return int(a.value), int(b.value)

    def match_probed(self, state: torch.Tensor, keys: torch.Tensor, blk_off: torch.Tensor, n_blocks: int,
                     matched: torch.Tensor | None = None) -> torch.Tensor:
        R = blk_off.numel() - 1
        if matched is None:
            matched = torch.empty((max(R, 1), self.n_instances), dtype=torch.int32, device=keys.device)
        _check("smetric_match_probed", _lib.smetric_match_probed(
            self.ref, C.c_void_p(state.data_ptr()), state.numel(), _dev(keys, torch.uint64, "keys"),
            _dev(blk_off, torch.int64, "blk_off"), R, n_blocks, _dev(matched, torch.int32, "matched"), _stream()))
        return matched[:R]

    def insert_probed(self, state: torch.Tensor, n_req: int, n_blocks: int, instance: torch.Tensor,
                      session: torch.Tensor, epoch: int, workspace: torch.Tensor | None = None):
        ws = self._workspace(insert_ws_bytes(n_blocks)) if workspace is None else workspace
        sess = _dev(session, torch.int32, "session") if session.dtype == torch.int32 else _dev(session, torch.uint32, "session")
        _check("smetric_index_insert_probed", _lib.smetric_index_insert_probed(
            self.ref, C.c_void_p(state.data_ptr()), state.numel(), n_req, n_blocks,
            _dev(instance, torch.int32, "instance"), sess, C.c_uint32(epoch), C.c_void_p(ws.data_ptr()), ws.numel(),
            _stream()))

    def snapshot(self, out: torch.Tensor | None = None) -> torch.Tensor:
        """A device copy of the whole index (attach it, or restore from it)."""
        if out is None:
            return self.mem.clone()
        out.copy_(self.mem)
        return out

    def restore(self, snap: torch.Tensor):
        self.mem.copy_(snap)
