"""The throughput configuration at full size on the GPU, in the launch configuration
bench.py times: 1,024 instances, one batch of 16,384 requests (~481M tokens, ~30M
blocks) against a 200M-entry index in 2^28 slots (~0.75 occupied) -- the prior turns of
four batches on uniform home instances, padded with filler keys that match nothing.

Checks: a sample of the batch's requests bit for bit (keys, matched rows, targets,
branches) against the oracle run on the exact restriction of the index to their keys
(their own prior turn on its home, and every prior turn's copy of the shared prefix they
use); then the product path's insert at the targets, by what it must satisfy on a
prefix-closed index: exactly the distinct new (key, target) pairs are added, and every
request then sees its whole prompt on its target (Sec. 2 append-only prompts; Sec. 4.2
the target caches what it prefills)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_08565_amd import workload as W
from tests.parity import check_probed_insert_full, say, to_dev

pytestmark = pytest.mark.gpu

ENTRIES = 200_000_000
SLOTS = 1 << 28
PRIOR_BATCHES = 4  # batch 0 is routed; batches 0..3 have their prior turns in the index


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _prior_keys(S, keys, blk_off, prior_len):
    prior_blocks = (prior_len // W.BLOCK).astype(np.int64)
    pos = np.repeat(blk_off[:-1] - np.concatenate([[0], np.cumsum(prior_blocks)[:-1]]), prior_blocks) + np.arange(
        int(prior_blocks.sum()))
    pk = keys.view(torch.int64)[to_dev(pos)].view(torch.uint64).contiguous()
    poff = np.zeros(len(prior_blocks) + 1, np.int64)
    poff[1:] = np.cumsum(prior_blocks)
    return pk, poff


def test_throughput_config_full_size():
    from paper_2607_08565_amd import smetric as S
    tw = W.ThroughputWorkload()
    I = tw.n_inst
    tbs = [tw.batch(b) for b in range(PRIOR_BATCHES)]
    b0 = tbs[0].batch
    blk0, nb0 = S.block_offsets(b0.tok_off)
    cap = ENTRIES + nb0
    gix = S.Index(cap, I, n_slots=SLOTS)
    ws = torch.empty(S.insert_ws_bytes(max(nb0, 16_000_000)), dtype=torch.uint8, device="cuda")
    for tb in tbs:
        bt = tb.batch
        blk, nb = S.block_offsets(bt.tok_off)
        keys = S.hash_blocks(to_dev(bt.tokens), to_dev(bt.tok_off), to_dev(blk), nb)
        pk, poff = _prior_keys(S, keys, blk, tb.prior_len)
        gix.insert(pk, to_dev(poff), int(poff[-1]), to_dev(tb.home), to_dev(bt.session), 0, workspace=ws)
        del keys, pk
    n_prior, st = gix.stats()
    assert st == 0
    done, c = n_prior, 0
    while done < ENTRIES:  # filler, 64 entries per instance group
        m = min(16_000_000, ENTRIES - done)
        fk, fi, fs = tw.filler(m, chunk=c)
        R = (m + 63) // 64
        off = np.minimum(np.arange(R + 1, dtype=np.int64) * 64, m)
        gix.insert(to_dev(fk), to_dev(off), m, to_dev(fi[::64][:R].copy()), to_dev(fs[:R].copy()), 0, workspace=ws)
        done += m
        c += 1
    n, st = gix.stats()
    assert st == 0 and n == ENTRIES, (n, st)
    say(f"  index: {n_prior} prior-turn entries + filler = {n} in {gix.n_slots} slots "
        f"(occupancy {n / gix.n_slots:.3f})")
    # the batch, as bench.py runs it
    d_boff = to_dev(blk0)
    keys, state = gix.hash_partition(to_dev(b0.tokens), to_dev(b0.tok_off), d_boff, nb0)
    gix.probe_lookup(state, keys, d_boff, nb0)
    gm = gix.match_probed(state, keys, d_boff, nb0).cpu().numpy()
    gt, gb = S.route(to_dev(gm), to_dev(b0.prompt_len), to_dev(b0.hist_len), to_dev(b0.turn), to_dev(b0.q),
                     W.DEFAULT_PARAMS, b0.rr_base)
    gt, gb = gt.cpu().numpy(), gb.cpu().numpy()
    say(f"  batch: {b0.n_req} requests, {nb0} blocks, branches {np.bincount(gb, minlength=5).tolist()}")
    # sampled parity against the oracle on the restriction of the index to the sample's keys
    rng = np.random.default_rng(104)
    sample = np.sort(rng.choice(b0.n_req, 48, replace=False))
    parts = [b0.tokens[b0.tok_off[s]: b0.tok_off[s + 1]] for s in sample]
    toff = np.zeros(len(sample) + 1, np.int64)
    toff[1:] = np.cumsum([len(p) for p in parts])
    ob, ok = oracle.hash_blocks(np.concatenate(parts), toff, W.BLOCK, W.DEFAULT_SEED)
    gk = keys[:nb0].cpu().numpy()
    for i, s in enumerate(sample):
        assert np.array_equal(gk[blk0[s]: blk0[s + 1]], ok[ob[i]: ob[i + 1]]), f"keys of request {s}"
    oix = oracle.Index(1 << 40, I)
    tb0 = tbs[0]
    prior = (tb0.prior_len[sample] // W.BLOCK).astype(np.int64)
    segs = [ok[ob[i]: ob[i] + prior[i]] for i in range(len(sample))]
    inst = list(tb0.home[sample])
    P = len(tw.prefixes[0])
    for p in np.unique(tb0.prefix_of[sample]):
        _, pk = oracle.hash_blocks(tw.prefixes[p], [0, P], W.BLOCK, W.DEFAULT_SEED)
        for tb in tbs:
            for s in np.nonzero(tb.prefix_of == p)[0]:
                m = int(min(tb.prior_len[s], P, tb.batch.prompt_len[s]) // W.BLOCK)
                if m:
                    segs.append(pk[:m])
                    inst.append(tb.home[s])
    soff = np.zeros(len(segs) + 1, np.int64)
    soff[1:] = np.cumsum([len(x) for x in segs])
    assert oix.insert(np.concatenate(segs), soff, np.asarray(inst, np.int32), np.zeros(len(segs), np.uint32), 0) == 0
    om = oix.match(ok, ob)
    for i, s in enumerate(sample):
        assert np.array_equal(gm[s], om[i]), f"matched row of request {s}"
        ot, obr = oracle.route(om[i: i + 1], b0.prompt_len[s: s + 1], b0.hist_len[s: s + 1], b0.turn[s: s + 1],
                               b0.q, W.DEFAULT_PARAMS, b0.rr_base + int(s))
        assert gt[s] == ot[0] and gb[s] == obr[0], f"decision of request {s}"
    say(f"  {len(sample)} sampled requests bit-exact ({oix.size} restricted oracle entries)")
    added = check_probed_insert_full(gix, b0, blk0, nb0, keys, state, gm, gt)
    assert 5_000_000 < added < nb0
