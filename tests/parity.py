"""Shared driver for GPU-vs-oracle parity: runs a batch sequence through the HIP library
and through the CPU oracle side by side.  Each side consumes only its own outputs; every
block key, matched-prefix row, target, branch and the sorted index dump are compared
bit for bit after every step."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2607_08565_amd import workload as W


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


class Pair:
    """The GPU path and the oracle holding the same index state."""

    def __init__(self, capacity: int, n_inst: int, seed: int = W.DEFAULT_SEED, block: int = W.BLOCK,
                 n_slots: int = 0):
        from paper_2607_08565_amd import smetric as S
        self.S = S
        self.I, self.seed, self.B = n_inst, seed, block
        self.gix = S.Index(capacity, n_inst, n_slots=n_slots)
        self.oix = oracle.Index(capacity, n_inst)

    def hash_both(self, tokens, tok_off):
        S = self.S
        blk_off, nb = S.block_offsets(tok_off, self.B)
        d_tok = to_dev(tokens if len(tokens) else np.zeros(1, np.int32))
        d_toff, d_boff = to_dev(tok_off), to_dev(blk_off)
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        keys = S.hash_blocks(d_tok, d_toff, d_boff, nb, self.B, self.seed, status=status)
        ob, ok = oracle.hash_blocks(tokens, tok_off, self.B, self.seed)
        assert np.array_equal(ob, blk_off), "block offsets"
        gk = keys[:nb].cpu().numpy()
        assert int(status.item()) == 0
        bad = np.nonzero(gk != ok)[0]
        assert len(bad) == 0, f"{len(bad)} key mismatches, first at block {bad[:5]}"
        return d_boff, nb, keys, ok, blk_off

    def insert_both(self, d_keys, d_boff, nb, okeys, blk_off, inst, sess, epoch):
        self.gix.insert(d_keys, d_boff, nb, to_dev(np.asarray(inst, np.int32)), to_dev(np.asarray(sess, np.uint32)), epoch)
        rc = self.oix.insert(okeys, blk_off, inst, sess, epoch)
        return rc

    def compare_index(self, what=""):
        n, st = self.gix.stats()
        assert n == self.oix.size, f"{what}: entry count gpu {n} oracle {self.oix.size}"
        assert st == self.oix.status, f"{what}: status gpu {st} oracle {self.oix.status}"
        gk, gv = self.gix.dump()
        ok, ov = self.oix.dump()
        assert np.array_equal(gk, ok), f"{what}: dumped keys differ"
        bad = np.nonzero(gv != ov)[0]
        assert len(bad) == 0, f"{what}: {len(bad)} dumped values differ, e.g. {[(hex(gv[i]), hex(ov[i])) for i in bad[:3]]}"

    def step(self, batch: W.Batch, params=None, rr_base=None, check_dump=True, what="", probed=False):
        """hash -> match -> route -> insert at target; returns (targets, branches).
        probed: the region-ordered path (probe once; match and insert from the probe state)."""
        params = params or W.DEFAULT_PARAMS
        rr = batch.rr_base if rr_base is None else rr_base
        d_boff, nb, d_keys, okeys, blk_off = self.hash_both(batch.tokens, batch.tok_off)
        state = None
        if probed:
            state = self.gix.probe(d_keys, d_boff, nb)
            gm = self.gix.match_probed(state, d_keys, d_boff, nb)
        else:
            gm = self.gix.match(d_keys, d_boff, nb)
        om = self.oix.match(okeys, blk_off)
        g = gm.cpu().numpy()
        bad = np.argwhere(g != om)
        assert len(bad) == 0, f"{what}: {len(bad)} matched mismatches, first (r,i)={bad[:3].tolist()} gpu={[g[tuple(x)] for x in bad[:3]]} orc={[om[tuple(x)] for x in bad[:3]]}"
        gt, gb = self.S.route(gm, to_dev(batch.prompt_len), to_dev(batch.hist_len), to_dev(batch.turn),
                              to_dev(batch.q), params, rr)
        ot, ob = oracle.route(om, batch.prompt_len, batch.hist_len, batch.turn, batch.q, params, rr)
        gt, gb = gt.cpu().numpy(), gb.cpu().numpy()
        assert np.array_equal(gt, ot), f"{what}: targets differ at {np.nonzero(gt != ot)[0][:5]}"
        assert np.array_equal(gb, ob), f"{what}: branches differ at {np.nonzero(gb != ob)[0][:5]}"
        if probed:
            self.gix.insert_probed(state, batch.n_req, nb, to_dev(np.asarray(ot, np.int32)),
                                   to_dev(np.asarray(batch.session, np.uint32)), batch.epoch)
            rc = self.oix.insert(okeys, blk_off, ot, batch.session, batch.epoch)
        else:
            rc = self.insert_both(d_keys, d_boff, nb, okeys, blk_off, ot, batch.session, batch.epoch)
        assert rc == 0, f"{what}: oracle insert rc {rc}"
        if check_dump:
            self.compare_index(what)
        return ot, ob


def run_sessions(wl: W.SessionWorkload, n_batches: int, capacity: int, evict: tuple[int, int] | None = None,
                 probed: bool = False, n_slots: int = 0):
    """Batch t = turn t of every session.  Open-loop workloads (with a placement) first
    enter turn t-1 on its placed instance; closed-loop ones rely on the post-route insert."""
    pair = Pair(capacity, wl.n_inst, n_slots=n_slots)
    prev_targets = None
    branches = []
    for t in range(n_batches):
        if wl.placement is not None and t > 0:
            prevb = wl.batch(t - 1)
            d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(prevb.tokens, prevb.tok_off)
            assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, wl.placement[t - 1], prevb.session, t - 1) == 0
        b = wl.batch(t, prev_targets)
        say(f"  batch {t}: R={b.n_req} tokens={b.n_tokens}")
        tg, br = pair.step(b, what=f"batch {t}", probed=probed)
        branches.append(br)
        prev_targets = tg
        if evict is not None:
            pair.gix.evict(*evict)
            assert pair.oix.evict(*evict) == 0
            pair.compare_index(f"batch {t} after evict")
    return pair, np.concatenate(branches)


def distinct_new_pairs(keys_h, blk_off_h, matched_h, target_h) -> int:
    """Distinct pairs (key_j of request r, target_r) with j >= matched[r][target_r]: the
    entries an insert at the targets adds to an index that is prefix-closed on every
    instance (each instance holds whole prompt prefixes), where the target holds exactly
    the request's first matched[r][target_r] blocks."""
    nb = np.diff(blk_off_h)
    R = len(nb)
    c_t = matched_h[np.arange(R), target_h].astype(np.int64)
    starts, cnt = blk_off_h[:-1] + c_t, nb - c_t
    base = np.concatenate([[0], np.cumsum(cnt)[:-1]]).astype(np.int64)
    pos = np.repeat(starts - base, cnt) + np.arange(int(cnt.sum()))
    k = keys_h[pos]
    t = np.repeat(np.asarray(target_h, np.uint64), cnt)
    o = np.lexsort((t, k))
    ks, ts = k[o], t[o]
    return int(len(ks) > 0) + int(np.count_nonzero((ks[1:] != ks[:-1]) | (ts[1:] != ts[:-1])))


def check_probed_insert_full(gix, batch: W.Batch, blk_off_h, nb: int, keys, state, matched_h, target_h):
    """A full-size check of the product path's post-route insert (smetric_index_insert_probed)
    that needs no full oracle, on an index that is prefix-closed on every instance and not
    evicted: (i) the entry count grows by exactly the distinct new (key, target) pairs, and
    (ii) matching the same batch again gives matched[r][target[r]] = its block count for every
    request (Sec. 2: prompts are append-only; Sec. 4.2: the target caches what it prefills)."""
    R = batch.n_req
    n0, st = gix.stats()
    assert st == 0
    expect = distinct_new_pairs(keys[:nb].cpu().numpy(), blk_off_h, matched_h, target_h)
    gix.insert_probed(state, R, nb, to_dev(np.asarray(target_h, np.int32)),
                      to_dev(np.asarray(batch.session, np.uint32)), batch.epoch)
    n1, st = gix.stats()
    assert st == 0, f"insert status {st}"
    assert n1 - n0 == expect, f"insert added {n1 - n0} entries, expected {expect} distinct new pairs"
    d_boff = to_dev(blk_off_h)
    keys2, state2 = gix.hash_partition(to_dev(batch.tokens), to_dev(batch.tok_off), d_boff, nb)
    gix.probe_lookup(state2, keys2, d_boff, nb)
    m2 = gix.match_probed(state2, keys2, d_boff, nb).cpu().numpy()
    whole = m2[np.arange(R), np.asarray(target_h, np.int64)] == np.diff(blk_off_h)
    assert whole.all(), f"{int((~whole).sum())} requests do not see their whole prompt on their target"
    say(f"  insert checked at full size: +{n1 - n0} entries ({n1} total), every request whole on its target")
    return n1 - n0
