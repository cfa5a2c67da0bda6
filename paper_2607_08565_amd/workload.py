"""Seeded synthetic agent-serving workloads.

This module only draws inputs -- token IDs, prompt lengths, shared-prefix choices,
placements and instance loads -- for the matching/routing path.  It holds none of the
method's arithmetic (no block split, hashing, matching or routing), so the GPU library
and the CPU oracle can both be fed from it without sharing any computation.

Shapes follow the paper's workload description: append-only agent sessions in which
turn t's prompt extends turn t-1's (Sec. 2, "Agentic workflow and the agent session"),
shared system prompts that serve first turns (Sec. 3.1, Finding 3), reuse above 80 %
(Sec. 3.1, Finding 1), and long coding-agent prompts.  The paper's own traces are
private, so the five configurations below are synthetic stand-ins with those shapes.

Random streams: numpy ``Generator(PCG64(SeedSequence([base, k, stream, ...])))`` with
separate streams for tokens, lengths, prefix choice, placement, load and filler.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

VOCAB = 151936                   # token IDs are uniform in [0, VOCAB)
BLOCK = 16                       # tokens per KV$ block
DEFAULT_SEED = 0x534D4554524943  # "SMETRIC" in ASCII, the hash seed
Q_UNIT_NS = 20_000_000           # queued prefill time per unit of instance load (20 ms)
BASE_SEED = 0x5EED0000

# Route constants in integer nanoseconds of prefill time.  The TTFT budget b = 1 s and
# a = 62.5 ms per 1K prompt tokens are the paper's evaluation values (Sec. 5.2); the
# Eq. (1) coefficients, SLACK and HIT_RATIO are synthetic (the paper fits or tunes them
# without printing values): 10k tokens/s linear cost, 3 ns/token^2 attention cost,
# SLACK = 1 (inside the robust range 0.5-2 of Sec. 5.5), HIT_RATIO = 1/2 ("below one").
DEFAULT_PARAMS = dict(
    c_lin=100_000, c_att=3, slo_b=1_000_000_000, slo_a=62_500,
    slack_num=1, slack_den=1, hit_num=1, hit_den=2, block_size=BLOCK,
)

# Named RNG streams.
S_TOK, S_LEN, S_PREFIX, S_PLACE, S_LOAD, S_FILL, S_PREFIXTOK, S_DECODE, S_TRACE = range(9)

# Per-instance decode state for the colocated rule: the value of a slack meaning "no live
# decode" (any value >= it).
NO_DECODE = 1 << 62


def _rng(cfg: int, stream: int, *extra: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([BASE_SEED + cfg, stream, *extra])))


def zipf_choice(rng: np.random.Generator, n_items: int, s: float, size: int) -> np.ndarray:
    """Item k (0-based) drawn with probability proportional to (k+1)^-s."""
    p = np.arange(1, n_items + 1, dtype=np.float64) ** (-s)
    p /= p.sum()
    return rng.choice(n_items, size=size, p=p)


def uniform_tokens(rng: np.random.Generator, n: int) -> np.ndarray:
    return rng.integers(0, VOCAB, size=n, dtype=np.int32)


@dataclass
class Batch:
    """One routing batch: R prompts in CSR form plus the per-request route inputs."""
    tokens: np.ndarray        # int32[T]
    tok_off: np.ndarray       # int64[R+1]
    prompt_len: np.ndarray    # int32[R]
    hist_len: np.ndarray      # int32[R]  expected hit from history (previous prompt length)
    turn: np.ndarray          # int32[R]  0 = first turn
    session: np.ndarray       # uint32[R]
    q: np.ndarray             # int64[I]  queued prefill ns per instance
    rr_base: int = 0
    epoch: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def n_req(self) -> int:
        return len(self.tok_off) - 1

    @property
    def n_tokens(self) -> int:
        return int(self.tok_off[-1])


def _csr(prompts: list[np.ndarray]) -> tuple[np.ndarray, np.ndarray]:
    lens = np.array([len(p) for p in prompts], np.int64)
    off = np.zeros(len(prompts) + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    toks = np.concatenate(prompts).astype(np.int32) if prompts else np.zeros(0, np.int32)
    return toks, off


# ---------------------------------------------------------------------------------------
# Session workloads: each session owns one token stream; turn t's prompt is the first
# L_t tokens of it, so every turn extends the previous one.
# ---------------------------------------------------------------------------------------
class SessionWorkload:
    """Sessions x turns; batch t holds turn t of every session."""

    def __init__(self, cfg: int, n_inst: int, n_sess: int, n_turns: int, lens: np.ndarray,
                 streams: list[np.ndarray], load: str, placement: np.ndarray | None = None):
        self.cfg = cfg
        self.n_inst = n_inst
        self.n_sess = n_sess
        self.n_turns = n_turns
        self.lens = lens            # int64[n_turns, n_sess]
        self.streams = streams      # per-session token stream, length >= lens[-1, s]
        self.load = load            # "uniform100", "poisson50", "prev_counts"
        self.placement = placement  # optional int32[n_turns, n_sess]: open-loop placement of turn t
        self.prefix_of = None       # optional int64[n_sess]: shared prefix of each session (-1: none)

    def batch(self, t: int, prev_targets: np.ndarray | None = None) -> Batch:
        L = self.lens[t]
        toks, off = _csr([self.streams[s][: L[s]] for s in range(self.n_sess)])
        hist = self.lens[t - 1] if t > 0 else np.zeros(self.n_sess, np.int64)
        rl = _rng(self.cfg, S_LOAD, t)
        if self.load == "uniform100":
            q = rl.integers(0, 101, size=self.n_inst).astype(np.int64) * Q_UNIT_NS
        elif self.load == "poisson50":
            q = rl.poisson(50, size=self.n_inst).astype(np.int64) * Q_UNIT_NS
        elif self.load == "prev_counts":
            cnt = np.zeros(self.n_inst, np.int64)
            if prev_targets is not None:
                np.add.at(cnt, prev_targets[prev_targets >= 0], 1)
            q = cnt * Q_UNIT_NS
        else:
            raise ValueError(self.load)
        return Batch(tokens=toks, tok_off=off, prompt_len=L.astype(np.int32), hist_len=hist.astype(np.int32),
                     turn=np.full(self.n_sess, t, np.int32), session=np.arange(self.n_sess, dtype=np.uint32),
                     q=q, rr_base=t * self.n_sess, epoch=t)


def _streams_with_prefix(cfg: int, n_sess: int, total: np.ndarray, prefix_of: np.ndarray,
                         prefixes: list[np.ndarray]) -> list[np.ndarray]:
    out = []
    rt = _rng(cfg, S_TOK)
    for s in range(n_sess):
        pre = prefixes[prefix_of[s]] if prefix_of[s] >= 0 else np.zeros(0, np.int32)
        n_priv = max(int(total[s]) - len(pre), 0)
        out.append(np.concatenate([pre, uniform_tokens(rt, n_priv)]))
    return out


def config0(n_sess: int = 64, n_turns: int = 4, n_inst: int = 8, l0: int = 1024,
            app: tuple[int, int] = (128, 1024), prefix_len: int = 512, prefix_frac: float = 0.25) -> SessionWorkload:
    """Tiny trace: 8 instances, 64 sessions x 4 turns.  Turn 0 is 1,024 uniform tokens, each
    later turn appends U{128..1024}; a quarter of the sessions start with one shared
    512-token system prefix.  Before batch t the index holds turns < t, each placed on a
    uniform-random instance (open loop).  Loads are U{0..100} units."""
    cfg = 0
    rl = _rng(cfg, S_LEN)
    lens = np.zeros((n_turns, n_sess), np.int64)
    lens[0] = l0
    for t in range(1, n_turns):
        lens[t] = lens[t - 1] + rl.integers(app[0], app[1] + 1, size=n_sess)
    prefix = uniform_tokens(_rng(cfg, S_PREFIXTOK), prefix_len)
    n_pref = int(round(prefix_frac * n_sess))
    prefix_of = np.full(n_sess, -1, np.int64)
    prefix_of[_rng(cfg, S_PREFIX).permutation(n_sess)[:n_pref]] = 0
    streams = _streams_with_prefix(cfg, n_sess, lens[-1], prefix_of, [prefix])
    placement = _rng(cfg, S_PLACE).integers(0, n_inst, size=(n_turns, n_sess)).astype(np.int32)
    wl = SessionWorkload(cfg, n_inst, n_sess, n_turns, lens, streams, "uniform100", placement)
    wl.prefix_of = prefix_of
    return wl


def config1(n_sess: int = 4096, n_turns: int = 10, n_inst: int = 64, l0: int = 4096,
            app: tuple[int, int] = (256, 4096), cap: int = 65536, n_prefix: int = 16,
            prefix_len: int = 2048) -> SessionWorkload:
    """Mid agent fleet: 64 instances, 4,096 sessions x 10 turns.  Turn 0 is 4,096 tokens:
    one of 16 distinct 2,048-token system prefixes (Zipf 1.1) plus uniform tokens; turns
    grow by U{256..4096} tokens, capped at 65,536.  Closed loop from an empty index, one
    request per session per batch; loads Poisson(50) units."""
    cfg = 1
    rl = _rng(cfg, S_LEN)
    lens = np.zeros((n_turns, n_sess), np.int64)
    lens[0] = l0
    for t in range(1, n_turns):
        lens[t] = np.minimum(cap, lens[t - 1] + rl.integers(app[0], app[1] + 1, size=n_sess))
    rp = _rng(cfg, S_PREFIXTOK)
    prefixes = [uniform_tokens(rp, prefix_len) for _ in range(n_prefix)]
    prefix_of = zipf_choice(_rng(cfg, S_PREFIX), n_prefix, 1.1, n_sess)
    streams = _streams_with_prefix(cfg, n_sess, lens[-1], prefix_of, prefixes)
    wl = SessionWorkload(cfg, n_inst, n_sess, n_turns, lens, streams, "poisson50")
    wl.prefix_of = prefix_of
    return wl


def config2(n_sess: int = 1024, n_turns: int = 30, n_inst: int = 256, l0: int = 16384,
            app: tuple[int, int] = (512, 8192), cap: int = 131072, n_prefix: int = 4,
            prefix_len: int = 8192) -> SessionWorkload:
    """Long-context coding agent: 256 instances, 1,024 sessions x 30 turns.  Turn 0 is
    16,384 tokens including one of 4 shared 8,192-token tool/system prefixes (uniform);
    appends U{512..8192}, capped at 131,072.  Closed loop; each instance's load is the
    number of requests routed to it in the previous batch."""
    cfg = 2
    rl = _rng(cfg, S_LEN)
    lens = np.zeros((n_turns, n_sess), np.int64)
    lens[0] = l0
    for t in range(1, n_turns):
        lens[t] = np.minimum(cap, lens[t - 1] + rl.integers(app[0], app[1] + 1, size=n_sess))
    rp = _rng(cfg, S_PREFIXTOK)
    prefixes = [uniform_tokens(rp, prefix_len) for _ in range(n_prefix)]
    prefix_of = _rng(cfg, S_PREFIX).integers(0, n_prefix, size=n_sess)
    streams = _streams_with_prefix(cfg, n_sess, lens[-1], prefix_of, prefixes)
    wl = SessionWorkload(cfg, n_inst, n_sess, n_turns, lens, streams, "prev_counts")
    wl.prefix_of = prefix_of
    return wl


def config3(n_sess: int = 8192, n_turns: int = 8, n_inst: int = 128, prefix_len: int = 32768,
            tail: tuple[int, int] = (1024, 16384), app: int = 512) -> SessionWorkload:
    """Divergent shared-prefix stress: 128 instances, 8,192 sessions all sharing one
    32,768-token prefix, each with its own U{1024..16384}-token tail; every turn appends
    512 tokens.  Closed loop with LRU eviction of 5 % of the entries after each batch's
    insert (index capacity at a 0.7 load factor of ~50M entries); loads Poisson(50)."""
    cfg = 3
    rl = _rng(cfg, S_LEN)
    lens = np.zeros((n_turns, n_sess), np.int64)
    lens[0] = prefix_len + rl.integers(tail[0], tail[1] + 1, size=n_sess)
    for t in range(1, n_turns):
        lens[t] = lens[t - 1] + app
    prefix = uniform_tokens(_rng(cfg, S_PREFIXTOK), prefix_len)
    streams = _streams_with_prefix(cfg, n_sess, lens[-1], np.zeros(n_sess, np.int64), [prefix])
    wl = SessionWorkload(cfg, n_inst, n_sess, n_turns, lens, streams, "poisson50")
    wl.prefix_of = np.zeros(n_sess, np.int64)
    return wl


def open_loop_placement(wl: SessionWorkload) -> np.ndarray:
    """int32[n_turns, n_sess]: a uniform-random instance for every turn of every session,
    for running a closed-loop configuration open loop (turn t entered on its placement
    before batch t + 1), which lets a request's exact index restriction be built without
    replaying the routing of every earlier batch."""
    return _rng(wl.cfg, S_PLACE, 1).integers(0, wl.n_inst, size=(wl.n_turns, wl.n_sess)).astype(np.int32)


def prefix_blocks(wl_cfg: int) -> int:
    """Length in blocks of the shared prefix every session of configurations 1-3 starts with."""
    return {1: 2048, 2: 8192, 3: 32768}[wl_cfg] // BLOCK


# ---------------------------------------------------------------------------------------
# Throughput workload: every batch holds distinct sessions whose prior turn (the first
# 70 % of each prompt's blocks) was placed on a home instance beforehand.
# ---------------------------------------------------------------------------------------
@dataclass
class ThroughputBatch:
    batch: Batch
    home: np.ndarray          # int32[R]  instance holding the session's prior turn
    prior_len: np.ndarray     # int64[R]  tokens of the prior turn (a multiple of BLOCK)
    prefix_of: np.ndarray     # int64[R]  shared prefix id


class ThroughputWorkload:
    """Throughput max: 1,024 instances, 16,384 requests per batch, prompt lengths
    lognormal(median 24,576, sigma 0.6) clipped to [1,024, 131,072].  70 % of each prompt's
    blocks are its session's prior turn, which starts with one of 64 shared 4,096-token
    prefixes (Zipf 1.2); the rest are new uniform tokens.  Prior turns are placed on
    uniform-random home instances; the index is padded with filler entries (random keys,
    never matched) up to the target entry count.  Loads Poisson(50) units."""

    def __init__(self, n_req: int = 16384, n_inst: int = 1024, median: float = 24576.0, sigma: float = 0.6,
                 lmin: int = 1024, lmax: int = 131072, n_prefix: int = 64, prefix_len: int = 4096,
                 zipf_s: float = 1.2, prior_frac: float = 0.7, cfg: int = 4):
        self.cfg = cfg
        self.n_req = n_req
        self.n_inst = n_inst
        self.median, self.sigma, self.lmin, self.lmax = median, sigma, lmin, lmax
        self.prior_frac = prior_frac
        self.n_prefix = n_prefix
        rp = _rng(cfg, S_PREFIXTOK)
        self.prefixes = [uniform_tokens(rp, prefix_len) for _ in range(n_prefix)]
        self.zipf_s = zipf_s

    def batch(self, b: int) -> ThroughputBatch:
        R = self.n_req
        rl = _rng(self.cfg, S_LEN, b)
        L = np.clip(np.rint(rl.lognormal(np.log(self.median), self.sigma, size=R)), self.lmin, self.lmax).astype(np.int64)
        prior_blocks = np.floor(self.prior_frac * (L // BLOCK)).astype(np.int64)
        prior_len = prior_blocks * BLOCK
        prefix_of = zipf_choice(_rng(self.cfg, S_PREFIX, b), self.n_prefix, self.zipf_s, R)
        home = _rng(self.cfg, S_PLACE, b).integers(0, self.n_inst, size=R).astype(np.int32)
        off = np.zeros(R + 1, np.int64)
        np.cumsum(L, out=off[1:])
        toks = uniform_tokens(_rng(self.cfg, S_TOK, b), int(off[-1]))
        for r in range(R):
            pre = self.prefixes[prefix_of[r]]
            n = min(len(pre), int(L[r]))
            toks[off[r]: off[r] + n] = pre[:n]
        q = _rng(self.cfg, S_LOAD, b).poisson(50, size=self.n_inst).astype(np.int64) * Q_UNIT_NS
        batch = Batch(tokens=toks, tok_off=off, prompt_len=L.astype(np.int32), hist_len=prior_len.astype(np.int32),
                      turn=np.ones(R, np.int32), session=(np.arange(R, dtype=np.int64) + b * R).astype(np.uint32),
                      q=q, rr_base=b * R, epoch=1 + b)
        return ThroughputBatch(batch=batch, home=home, prior_len=prior_len, prefix_of=prefix_of)

    def decode_state(self, b: int, idle_frac: float = 0.3, max_slack_ns: int = 3_000_000_000,
                     mean_running: float = 8.0):
        """Colocated fleet at batch b: per instance the smallest slack of its live decodes
        (ns; NO_DECODE for the idle_frac of instances without decodes, else uniform in
        [0, max_slack_ns)) and its request count (Poisson(mean_running))."""
        rd = _rng(self.cfg, S_DECODE, b)
        idle = rd.random(self.n_inst) < idle_frac
        slack = rd.integers(0, max_slack_ns, size=self.n_inst).astype(np.int64)
        slack[idle] = NO_DECODE
        n_run = rd.poisson(mean_running, size=self.n_inst).astype(np.int32)
        return slack, n_run

    def filler(self, n: int, chunk: int = 0):
        """n filler entries: random 64-bit keys (reserved values 0 and 2^64-1 excluded),
        uniform instances, session ids above every real session."""
        rf = _rng(self.cfg, S_FILL, chunk)
        keys = rf.integers(1, np.iinfo(np.uint64).max - 1, size=n, dtype=np.uint64, endpoint=False)
        inst = rf.integers(0, self.n_inst, size=n).astype(np.int32)
        sess = np.full(n, (1 << 24) - 1, np.uint32)
        return keys, inst, sess


@dataclass
class Trace:
    """An anonymised multi-session trace: requests in arrival order with their tokens,
    user and turn, plus the generator's ground truth (never an input of the method)."""
    tokens: np.ndarray      # int32, CSR by request
    tok_off: np.ndarray     # int64[R+1]
    user: np.ndarray        # uint32[R]
    turn: np.ndarray        # int32[R]
    true_session: np.ndarray  # int32[R] generator's session id
    true_parent: np.ndarray   # int32[R] generator's previous request of the session (-1: none)
    compacted: np.ndarray     # bool[R] prompt rewritten (no prefix relation to the previous turn)

    @property
    def n_req(self) -> int:
        return len(self.tok_off) - 1


def session_trace(n_users: int = 64, sessions_per_user: int = 4, turns: int = 6, l0: int = 2048,
                  prefix_len: int = 1024, app: tuple[int, int] = (256, 2048), p_compact: float = 0.05,
                  p_retry: float = 0.03, compact_len: int = 1024, seed: int = 0) -> Trace:
    """Synthetic trace with the shapes App. A relies on: each user runs several sessions,
    all starting with the user's own system prefix; each turn's prompt extends the previous
    one (reply + tool output, App. A) by U{app} tokens; a compaction turn (probability
    p_compact) replaces the prompt with a fresh summary of compact_len tokens; a retry
    (probability p_retry) resends a turn's exact prompt.  Sessions start at uniform times and
    their turns are spaced by exponential gaps; requests are sorted by arrival."""
    rg = _rng(9, S_TRACE, seed)
    prompts, users, turns_l, sess, parents, comp, times = [], [], [], [], [], [], []
    sid = 0
    for u in range(n_users):
        sys_prefix = uniform_tokens(rg, prefix_len)
        for _ in range(sessions_per_user):
            t_now = rg.uniform(0.0, 1000.0)
            prompt = np.concatenate([sys_prefix, uniform_tokens(rg, max(l0 - prefix_len, 0))])
            prev_idx = -1
            for t in range(turns):
                is_comp = False
                if t > 0:
                    if rg.random() < p_compact:
                        prompt = uniform_tokens(rg, compact_len)
                        is_comp = True
                    prompt = np.concatenate([prompt, uniform_tokens(rg, int(rg.integers(app[0], app[1] + 1)))])
                reps = 2 if rg.random() < p_retry else 1
                parent_of_turn = prev_idx  # a retry has the same parent as the original
                for _k in range(reps):
                    prompts.append(prompt)
                    users.append(u)
                    turns_l.append(t)
                    sess.append(sid)
                    parents.append(parent_of_turn)  # generator-local index, remapped below
                    comp.append(is_comp)
                    times.append(t_now)
                    prev_idx = len(prompts) - 1  # the next turn follows the latest send
                    t_now += rg.exponential(5.0) + 1e-6
            sid += 1
    order = np.argsort(np.asarray(times), kind="stable")
    rank = np.empty(len(order), np.int64)
    rank[order] = np.arange(len(order))
    toks, off = _csr([prompts[i] for i in order])
    par = np.asarray(parents, np.int64)[order]
    par = np.where(par >= 0, rank[np.maximum(par, 0)], -1).astype(np.int32)
    return Trace(tokens=toks, tok_off=off, user=np.asarray(users, np.uint32)[order],
                 turn=np.asarray(turns_l, np.int32)[order], true_session=np.asarray(sess, np.int32)[order],
                 true_parent=par, compacted=np.asarray(comp, bool)[order])
