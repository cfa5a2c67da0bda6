"""Benchmark: one step = hash -> match -> route -> insert over one routing batch.

Workload (the throughput configuration): 1,024 instances, 16,384 requests per batch,
prompt lengths lognormal(median 24,576, sigma 0.6) clipped to [1,024, 131,072], 70 % of
each prompt's blocks being its session's prior turn, 64 shared 4,096-token prefixes
chosen Zipf(1.2), loads Poisson(50) x 20 ms.

The start index is fixed and does not depend on --steps: the prior turns of a fixed set
of distinct batches (each on a uniform-random home instance), padded with never-matching
filler entries to exactly --index-entries (200M) entries, in a table of --slots (2^28)
slots, i.e. ~0.75 occupied, with capacity for one more batch of pairs.  Every step -- warm-
up and timed -- starts from that index: a device snapshot of it is restored, untimed,
before each step, so every timed step routes a batch of distinct, pre-inserted sessions
against the same index.  Each timed step is bracketed by device synchronisations; the
inputs of every batch are resident in HBM before timing starts.

After the timed steps the last timed batch is checked at full size: the post-route
insert leaves every request's whole block sequence on its target (the append-only
property: matched[r][target[r]] = its block count, found by matching the batch again),
and the entry count grows by exactly the distinct (key, target) pairs the targets did not
hold; with the CPU baseline, a sample of its requests is compared bit for bit with the
oracle.

Prints one JSON line (see the fields at the end of main()).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "requests routed/sec + prompt tokens matched/sec; achieved HBM GB/s vs peak"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=6)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--n-req", type=int, default=16384)
    ap.add_argument("--n-inst", type=int, default=1024)
    ap.add_argument("--index-entries", type=int, default=200_000_000,
                    help="entries in the index at the start of every step")
    ap.add_argument("--slots", type=int, default=1 << 28, help="slots of the index table")
    ap.add_argument("--distinct-batches", type=int, default=8,
                    help="distinct batches whose prior turns are in the start index; steps cycle over them")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle time budget for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--direct", action="store_true",
                    help="match and insert probe the index themselves instead of sharing one region-ordered probe")
    ap.add_argument("--overlap-path", action="store_true",
                    help="also measure the hash + probe path with the next batch's hash beside this batch's "
                         "lookup and match (two streams); off by default, so that a profile of the default run "
                         "averages each kernel over the timed steps' launches only")
    ap.add_argument("--overlap-step", action="store_true",
                    help="also measure whole steps with the next batch's hash + partition beside this batch's "
                         "lookup, match, route and insert (two streams, the index restored between steps)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after the timed steps, copy 1 GiB on the device (the counter runs' scale)")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="print the per-kernel summary of a rocprofv3 --kernel-trace run of this script and exit")
    ap.add_argument("--summarize-sq", nargs=2, metavar=("SQ_CSV", "BENCH_JSON"),
                    help="print the per-kernel instruction counts of a rocprofv3 --pmc run of this script with "
                         "the SQ counters (and the JSON line of that run, which gives the tokens per batch) and exit")
    ap.add_argument("--summarize-pmc", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "BENCH_JSON"),
                    help="write the traffic file from two rocprofv3 --pmc runs of this script (and the JSON "
                         "line of one of them, which names the workload) and exit")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM bytes per launch (rocprofv3 FETCH_SIZE/WRITE_SIZE), if present")
    return ap.parse_args()


class Setup:
    """Resident inputs, the fixed start index, its snapshot and reusable output buffers."""

    def __init__(self, args):
        import torch

        from paper_2607_08565_amd import smetric as S
        from paper_2607_08565_amd import workload as W

        self.S, self.W, self.torch = S, W, torch
        self.args = args
        self.n_distinct = args.distinct_batches
        self.tw = W.ThroughputWorkload(n_req=args.n_req, n_inst=args.n_inst)
        t0 = time.time()
        self.host = [self.tw.batch(b) for b in range(self.n_distinct)]
        log(f"[setup] generated {self.n_distinct} distinct batches in {time.time() - t0:.1f}s")
        self.dev = []
        for tb in self.host:
            b = tb.batch
            blk_off, nb = S.block_offsets(b.tok_off)
            self.dev.append(dict(
                tokens=torch.from_numpy(b.tokens).cuda(), tok_off=torch.from_numpy(b.tok_off).cuda(),
                blk_off=torch.from_numpy(blk_off).cuda(), blk_off_h=blk_off, n_blocks=nb,
                prompt_len=torch.from_numpy(b.prompt_len).cuda(), hist_len=torch.from_numpy(b.hist_len).cuda(),
                turn=torch.from_numpy(b.turn).cuda(), session=torch.from_numpy(b.session).cuda(),
                q=torch.from_numpy(b.q).cuda()))
        max_blocks = max(d["n_blocks"] for d in self.dev)
        self.keys = torch.empty(max_blocks, dtype=torch.uint64, device="cuda")
        self.keys2 = [self.keys, torch.empty(max_blocks, dtype=torch.uint64, device="cuda")]
        self.matched = torch.empty((args.n_req, args.n_inst), dtype=torch.int32, device="cuda")
        self.target = torch.empty(args.n_req, dtype=torch.int32, device="cuda")
        self.branch = torch.empty(args.n_req, dtype=torch.uint8, device="cuda")
        self.filler_chunk = 16_000_000
        self.ws = torch.empty(S.insert_ws_bytes(max(max_blocks, self.filler_chunk)), dtype=torch.uint8, device="cuda")
        self.probe_state = torch.empty(S.probe_ws_bytes(max_blocks), dtype=torch.uint8, device="cuda")
        self.state2 = [self.probe_state, torch.empty(S.probe_ws_bytes(max_blocks), dtype=torch.uint8, device="cuda")]
        # default-priority streams for the overlapped path measurement
        self.sA, self.sB = torch.cuda.Stream(), torch.cuda.Stream()
        # the start index: capacity for the start entries plus one batch of pairs, so the
        # insert's capacity pre-check always passes
        self.capacity = args.index_entries + max_blocks
        self.index = S.Index(self.capacity, args.n_inst, n_slots=args.slots)
        t0 = time.time()
        for tb, d in zip(self.host, self.dev):
            self._prepopulate(tb, d)
        n, st = self.index.stats()
        assert st == 0, f"index status {st} after prior turns"
        self.prior_entries = n
        if n > args.index_entries:
            raise SystemExit(f"{self.n_distinct} batches' prior turns give {n} entries, more than --index-entries")
        self._filler(args.index_entries - n)
        n, st = self.index.stats()
        assert st == 0 and n == args.index_entries, f"index status {st}, {n} entries after filler"
        self.start_entries = n
        self.snap = self.index.snapshot()
        torch.cuda.synchronize()
        log(f"[setup] index: {self.prior_entries} prior-turn entries + filler = {n} entries in {self.index.n_slots} "
            f"slots (occupancy {n / self.index.n_slots:.3f}, {self.index.mem.numel() / 2**30:.2f} GiB, "
            f"capacity {self.capacity}) in {time.time() - t0:.1f}s")

    def batch_of(self, i: int) -> int:
        """The batch that step i (warm-up steps first, then timed ones) routes."""
        return i % self.n_distinct

    def restore(self):
        self.index.restore(self.snap)

    def _prepopulate(self, tb, d):
        torch, S = self.torch, self.S
        keys = S.hash_blocks(d["tokens"], d["tok_off"], d["blk_off"], d["n_blocks"], keys=self.keys)
        prior_blocks = (tb.prior_len // self.W.BLOCK).astype(np.int64)
        starts = d["blk_off_h"][:-1]
        pos = np.repeat(starts - np.concatenate([[0], np.cumsum(prior_blocks)[:-1]]), prior_blocks) + np.arange(
            int(prior_blocks.sum()))
        pk = keys.view(torch.int64)[torch.from_numpy(pos).cuda()].view(torch.uint64).contiguous()
        poff = np.zeros(len(prior_blocks) + 1, np.int64)
        poff[1:] = np.cumsum(prior_blocks)
        self.index.insert(pk, torch.from_numpy(poff).cuda(), int(poff[-1]), torch.from_numpy(tb.home).cuda(),
                          d["session"], 0, workspace=self.ws)

    def _filler(self, n: int):
        torch = self.torch
        per = 64
        chunk = self.filler_chunk
        done, c = 0, 0
        while done < n:
            m = min(chunk, n - done)
            keys, inst, sess = self.tw.filler(m, chunk=c)
            R = (m + per - 1) // per
            off = np.minimum(np.arange(R + 1, dtype=np.int64) * per, m)
            self.index.insert(torch.from_numpy(keys).cuda(), torch.from_numpy(off).cuda(), m,
                              torch.from_numpy(inst[::per][:R].copy()).cuda(),
                              torch.from_numpy(sess[:R].copy()).cuda(), 0, workspace=self.ws)
            done += m
            c += 1

    CALLS = ("hash", "probe", "match", "route", "insert")
    # names in the JSON line: what each timed call is (region-ordered path)
    SHOW = {"hash": "hash_partition", "probe": "lookup", "match": "match", "route": "route", "insert": "insert"}

    def step(self, b: int, ev=None):
        """The timed unit: every call of the path on the current stream."""
        S, d, tb = self.S, self.dev[b], self.host[b]
        rec = (lambda k: ev[k].record()) if ev is not None else (lambda k: None)
        nb = d["n_blocks"]
        rec(0)
        if self.args.direct:
            S.hash_blocks(d["tokens"], d["tok_off"], d["blk_off"], nb, keys=self.keys)
        else:  # the block keys and the region partition in one call
            self.index.hash_partition(d["tokens"], d["tok_off"], d["blk_off"], nb, keys=self.keys,
                                      state=self.probe_state)
        rec(1)
        if not self.args.direct:
            self.index.probe_lookup(self.probe_state, self.keys, d["blk_off"], nb)
        rec(2)
        if self.args.direct:
            self.index.match(self.keys, d["blk_off"], nb, matched=self.matched)
        else:
            self.index.match_probed(self.probe_state, self.keys, d["blk_off"], nb, matched=self.matched)
        rec(3)
        S.route(self.matched, d["prompt_len"], d["hist_len"], d["turn"], d["q"], self.W.DEFAULT_PARAMS,
                tb.batch.rr_base, target=self.target, branch=self.branch)
        rec(4)
        if self.args.direct:
            self.index.insert(self.keys, d["blk_off"], nb, self.target, d["session"], tb.batch.epoch,
                              workspace=self.ws)
        else:
            self.index.insert_probed(self.probe_state, self.args.n_req, nb, self.target, d["session"],
                                     tb.batch.epoch, workspace=self.ws)
        rec(5)

    def path_only(self, b: int, p: int, matched):
        """Hash + partition, lookup and match of batch b into buffer set p (no route, no
        insert: the index is not changed)."""
        d, nb = self.dev[b], self.dev[b]["n_blocks"]
        self.index.hash_partition(d["tokens"], d["tok_off"], d["blk_off"], nb, keys=self.keys2[p],
                                  state=self.state2[p])
        self.index.probe_lookup(self.state2[p], self.keys2[p], d["blk_off"], nb)
        self.index.match_probed(self.state2[p], self.keys2[p], d["blk_off"], nb, matched=matched)

    def path_overlapped(self, batches, matched2):
        """The hash + probe path over consecutive batches on two default-priority streams:
        batch k+1's hash and partition (stream A; it reads no index contents) run beside
        batch k's lookup and match (stream B).  Buffer sets alternate, and a set is reused
        only after the match that read it has finished.  Returns the wall time."""
        torch = self.torch
        hashed, matched_done = {}, {}
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k, b in enumerate(batches):
            p = k % 2
            with torch.cuda.stream(self.sA):
                if k - 2 in matched_done:
                    self.sA.wait_event(matched_done[k - 2])
                d, nb = self.dev[b], self.dev[b]["n_blocks"]
                self.index.hash_partition(d["tokens"], d["tok_off"], d["blk_off"], nb, keys=self.keys2[p],
                                          state=self.state2[p])
                e = torch.cuda.Event()
                e.record(self.sA)
                hashed[k] = e
            with torch.cuda.stream(self.sB):
                self.sB.wait_event(hashed[k])
                self.index.probe_lookup(self.state2[p], self.keys2[p], d["blk_off"], nb)
                self.index.match_probed(self.state2[p], self.keys2[p], d["blk_off"], nb, matched=matched2[p])
                e = torch.cuda.Event()
                e.record(self.sB)
                matched_done[k] = e
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    def step_overlapped(self, batches):
        """Whole steps over consecutive batches with the next batch's hash and partition
        (stream A; it reads no index contents) beside this batch's lookup, match, route and
        insert (stream B), buffer sets alternating; the index is restored between steps,
        untimed, after both streams finished.  Batch 0's hash is timed alone.  Returns the
        timed seconds (one hash, lookup, match, route and insert per batch)."""
        torch = self.torch
        total = 0.0
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        with torch.cuda.stream(self.sA):
            d = self.dev[batches[0]]
            self.index.hash_partition(d["tokens"], d["tok_off"], d["blk_off"], d["n_blocks"], keys=self.keys2[0],
                                      state=self.state2[0])
        torch.cuda.synchronize()
        total += time.perf_counter() - t0
        for k, b in enumerate(batches):
            p, d, tb = k % 2, self.dev[b], self.host[b]
            nb = d["n_blocks"]
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            with torch.cuda.stream(self.sB):
                self.index.probe_lookup(self.state2[p], self.keys2[p], d["blk_off"], nb)
                self.index.match_probed(self.state2[p], self.keys2[p], d["blk_off"], nb, matched=self.matched)
                self.S.route(self.matched, d["prompt_len"], d["hist_len"], d["turn"], d["q"], self.W.DEFAULT_PARAMS,
                             tb.batch.rr_base, target=self.target, branch=self.branch)
                self.index.insert_probed(self.state2[p], self.args.n_req, nb, self.target, d["session"],
                                         tb.batch.epoch, workspace=self.ws)
            if k + 1 < len(batches):  # set 1 - p was last read by the previous step, which has finished
                with torch.cuda.stream(self.sA):
                    dn = self.dev[batches[k + 1]]
                    self.index.hash_partition(dn["tokens"], dn["tok_off"], dn["blk_off"], dn["n_blocks"],
                                              keys=self.keys2[1 - p], state=self.state2[1 - p])
            torch.cuda.synchronize()
            total += time.perf_counter() - t0
            self.restore()
            torch.cuda.synchronize()
        return total


# kernels each timed call launches, in order (names as rocprofv3 reports them)
CALL_KERNELS = {
    # smetric_hash_partition: the state cleared, the block keys (the hash itself taking the
    # region counts), each block's request, then the region partition's scan and scatter
    "hash": ["zero2_kernel", "hash16_kernel<8, true>", "req_of_kernel", "part_scan_kernel", "part_scatter_kernel"],
    # smetric_probe_lookup: each request's probe bound, then one holder descriptor per block,
    # in region order
    "probe": ["zero2_kernel", "bound_kernel", "probe_kernel<2>"],
    "match": ["match_kernel<1, true>"],
    "route": ["route_kernel<0>"],
    "insert": ["fill_kernel", "insp_valid_kernel", "insp_classify_kernel", "insp_size_kernel", "insp_bcount_kernel",
               "insp_bscan_kernel", "insp_size2_kernel", "insp_bscatter_kernel",
               "insp_bdedupe_kernel", "insp_check_kernel", "insp_place_kernel", "spill_kernel",
               "deferred_kernel"],
}


def _kname(full: str) -> str:
    """Kernel name as rocprofv3 prints it, without namespaces, return type and arguments."""
    n = full.replace("smk::(anonymous namespace)::", "")
    if n.startswith("void "):
        n = n[5:]
    depth = 0
    for i, ch in enumerate(n):  # cut at the argument list (the first '(' outside template brackets)
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return n[:i]
    return n


STEP_CALLS = [(c, k) for c in ("hash", "probe", "match", "route", "insert") for k in CALL_KERNELS[c]]
STEP_SEQ = [k for _, k in STEP_CALLS]


def timed_step_dispatches(rows, steps: int):
    """rows: (dispatch_id, kernel name, payload) in any order.  Returns the dispatches of the
    last `steps` occurrences of one whole step (its kernels in launch order), as a list of
    lists of (name, payload); set-up, warm-up and later measurements are left out."""
    rows = sorted(rows, key=lambda r: r[0])
    names = [r[1] for r in rows]
    L = len(STEP_SEQ)
    starts = [i for i in range(len(rows) - L + 1) if names[i:i + L] == STEP_SEQ]
    if len(starts) < steps:
        raise SystemExit(f"found {len(starts)} whole steps in the trace, expected {steps}")
    return [[(names[j], rows[j][2]) for j in range(i, i + L)] for i in starts[-steps:]]


def summarize_trace(csv_path: str, steps: int):
    """Markdown summary of a rocprofv3 --kernel-trace CSV: per-kernel durations over the
    timed steps of one bench.py run."""
    import csv
    rows = [(int(r["Dispatch_Id"]), _kname(r["Kernel_Name"]),
             (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3) for r in csv.DictReader(open(csv_path))]
    st = timed_step_dispatches(rows, steps)
    out = ["| call | kernel | mean µs | min µs | max µs |", "|---|---|---|---|---|"]
    per_call = {}
    for j, (c, k) in enumerate(STEP_CALLS):
        d = [s[j][1] for s in st]
        out.append(f"| {c} | {k} | {np.mean(d):.1f} | {min(d):.1f} | {max(d):.1f} |")
        per_call[c] = per_call.get(c, 0.0) + float(np.mean(d))
    out += ["", "| call | sum of kernel means µs |", "|---|---|"]
    out += [f"| {c} | {v:.1f} |" for c, v in per_call.items()]
    return "\n".join(out)


def workload_key(cfg: dict) -> dict:
    """What the counters depend on besides the kernel sources: the bench workload."""
    return {k: cfg[k] for k in ("n_instances", "requests_per_batch", "index_entries_start", "index_slots",
                                "index_capacity", "distinct_batches")}


def summarize_pmc(fetch_csv: str, write_csv: str, steps: int, copy_bytes: int, bench_json: str):
    """HBM traffic per timed call from two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE,
    KiB per dispatch), each scaled by what the counter reads for the 1 GiB device copy that
    --calibrate-copy issues after the timed steps (the smallest copy kernel of at least
    64 MiB in each run: the index snapshot and its restores are larger).
    The result is keyed to the kernel sources and to the workload named by the JSON line of
    one of the runs."""
    import csv

    def load(path, counter):
        rows, copies = [], []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            n, v = _kname(r["Kernel_Name"]), float(r["Counter_Value"]) * 1024.0
            rows.append((int(r["Dispatch_Id"]), n, v))
            if "copyBuffer" in n:
                copies.append((int(r["Dispatch_Id"]), v))
        # the calibration: the smallest copy of at least 1/16 of its size (the index
        # snapshot and its restores are larger copies, small ones are set-up transfers)
        big = [v for _, v in copies if v >= copy_bytes / 16]
        return rows, min(big) if big else 0.0

    fr, fcopy = load(fetch_csv, "FETCH_SIZE")
    wr, wcopy = load(write_csv, "WRITE_SIZE")
    if fcopy <= 0 or wcopy <= 0:
        raise SystemExit("no calibration copy in the counter runs (run bench.py with --calibrate-copy)")
    kf, kw = copy_bytes / fcopy, copy_bytes / wcopy
    fs, ws = timed_step_dispatches(fr, steps), timed_step_dispatches(wr, steps)
    line = [x for x in open(bench_json).read().splitlines() if x.startswith("{")][-1]
    cfg = json.loads(line)["config"]
    res = {"sources_sha256_16": kernel_sources_hash(), "workload": workload_key(cfg), "steps": steps,
           "fetch_scale": round(kf, 4), "write_scale": round(kw, 4), "kernels": {}}
    out = [f"Copy calibration: FETCH_SIZE x {kf:.3f}, WRITE_SIZE x {kw:.3f} = bytes of a {copy_bytes >> 20} MiB copy.",
           "", "| call | kernel | fetched MB | written MB | traffic MB |", "|---|---|---|---|---|"]
    for j, (c, k) in enumerate(STEP_CALLS):
        f = float(np.mean([s[j][1] for s in fs])) * kf
        w = float(np.mean([s[j][1] for s in ws])) * kw
        res["kernels"][f"{c}:{k}:{j}"] = round(f + w)
        res[c] = res.get(c, 0) + round(f + w)
        out.append(f"| {c} | {k} | {f / 1e6:.1f} | {w / 1e6:.1f} | {(f + w) / 1e6:.1f} |")
    out += ["", "| call | traffic MB per launch |", "|---|---|"]
    out += [f"| {c} | {res[c] / 1e6:.1f} |" for c in ("hash", "probe", "match", "route", "insert")]
    return res, "\n".join(out)


SQ_COUNTERS = ("SQ_WAVES", "SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_INSTS_LDS", "SQ_INSTS_VMEM_RD", "SQ_INSTS_VMEM_WR",
               "SQ_WAVE_CYCLES")


def summarize_sq(csv_path: str, steps: int, bench_json: str):
    """Per-kernel instruction counts over the timed steps from one rocprofv3 --pmc run with
    the SQ counters (wavefront instructions per launch; a VALU instruction covers 64 lanes),
    and the counting hash's VALU lane operations per prompt token."""
    import csv
    per = {c: [] for c in SQ_COUNTERS}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] in per:
            per[r["Counter_Name"]].append((int(r["Dispatch_Id"]), _kname(r["Kernel_Name"]), float(r["Counter_Value"])))
    st = {c: timed_step_dispatches(rows, steps) for c, rows in per.items() if rows}
    line = [x for x in open(bench_json).read().splitlines() if x.startswith("{")][-1]
    tokens = json.loads(line)["config"]["tokens_per_batch"]
    cols = [c for c in SQ_COUNTERS if c in st]
    out = ["| call | kernel | " + " | ".join(c[3:] for c in cols) + " |", "|---|---|" + "---|" * len(cols)]
    mean = {}
    for j, (c, k) in enumerate(STEP_CALLS):
        vals = {q: float(np.mean([s[j][1] for s in st[q]])) for q in cols}
        mean[(c, k)] = vals
        out.append(f"| {c} | {k} | " + " | ".join(f"{vals[q]:.4g}" for q in cols) + " |")
    hk = [key for key in mean if key[0] == "hash" and key[1].startswith("hash16_kernel")]
    if hk and "SQ_INSTS_VALU" in cols:
        v = mean[hk[0]]["SQ_INSTS_VALU"]
        out += ["", f"Counting hash: {v:.4g} VALU instructions x 64 lanes / {tokens:,} tokens = "
                    f"{v * 64 / tokens:.1f} VALU lane operations per token."]
    return "\n".join(out)


def kernel_sources_hash() -> str:
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2607_08565_amd", "csrc", "*"))):
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def algorithmic_bytes(setup, b, matched, I, n_probed=None, n_search=None):
    """Bytes the method itself must move for batch b (see the design notes):
    hash: 4 B per token read + 8 B per block key written;
    probe: 8 B key + one 64 B bucket burst per probe the lookup makes (the blocks before
    each request's probe bound, and its bound search; the match needs the blocks up to and
    including each request's first block nobody holds);
    match: the same 72 B per necessary block, I/8 B of holder bitmap per distinct block of a
    widely shared prefix probed in the batch (each bitmap is charged once), 4 B per
    (request, instance) written."""
    tb = setup.host[b]
    bt = tb.batch
    n_tok = int(bt.tok_off[-1])
    n_blk = int(setup.dev[b]["n_blocks"])
    nb = np.diff(setup.dev[b]["blk_off_h"])
    cmax = matched.max(axis=1)
    probes = np.minimum(cmax + 1, nb)  # blocks up to and including the first block nobody holds
    pre_blocks = len(setup.tw.prefixes[0]) // setup.W.BLOCK
    hot = np.minimum(probes, np.minimum(pre_blocks, nb))  # probed blocks of the request's shared prefix
    hot_distinct = int(sum(int(hot[tb.prefix_of == p].max(initial=0)) for p in range(len(setup.tw.prefixes))))
    R = len(nb)
    H = hot_distinct * (I // 8)
    hash_b = 4 * n_tok + 8 * n_blk
    match_b = int(probes.sum()) * (8 + 64) + H + 4 * R * I
    lookups = n_blk if n_probed is None else n_probed + n_search
    probe_b = lookups * (8 + 64)
    scan_b = int(probes.sum()) * 8 + H + 4 * R * I  # the match from descriptors: one per necessary block
    return dict(tokens=n_tok, blocks=n_blk, probes=int(probes.sum()), hot_probes=int(hot.sum()), lookups=lookups,
                blocks_probed=n_blk if n_probed is None else n_probed, search_probes=n_search or 0,
                hot_distinct=hot_distinct, H=H, descriptor=8 * n_blk, hash=hash_b, match=match_b, probe=probe_b,
                match_scan=scan_b, route=4 * R * I + 8 * I + 12 * R + 5 * R)


def cpu_baseline(setup, b: int, budget_s: float, gpu_out):
    """The oracle, as it stands, on a bounded sample of batch b: its first n requests,
    against the exact restriction of the start index to their keys (their own prior turns
    and every prior turn's copy of the shared prefixes they use; filler never matches),
    timed on one core.  Also checks the GPU's outputs of that batch for those requests bit
    for bit."""
    import oracle

    W = setup.W
    tw, hosts = setup.tw, setup.host
    tbs = hosts[b]
    bs = tbs.batch
    params = W.DEFAULT_PARAMS
    prefix_len = len(tw.prefixes[0])

    def run(n):
        R = n
        toks = bs.tokens[: bs.tok_off[R]]
        tok_off = bs.tok_off[: R + 1]
        ix = oracle.Index(1 << 40, tw.n_inst)
        # shared prefixes used by the sample, held by every session placed with them
        used = set(tbs.prefix_of[:R].tolist())
        for p in sorted(used):
            pre = tw.prefixes[p]
            pb, pk = oracle.hash_blocks(pre, [0, len(pre)], W.BLOCK, W.DEFAULT_SEED)
            for tb in hosts:
                sel = np.nonzero(tb.prefix_of == p)[0]
                for s in sel:
                    m = int(min(tb.prior_len[s], prefix_len) // W.BLOCK)
                    m = min(m, int(tb.batch.prompt_len[s]) // W.BLOCK)
                    if m:
                        ix.insert(pk[:m], [0, m], [tb.home[s]], [tb.batch.session[s]], 0)
        # the sample's own prior turns
        blk_off, keys = oracle.hash_blocks(toks, tok_off, W.BLOCK, W.DEFAULT_SEED)
        prior = (tbs.prior_len[:R] // W.BLOCK).astype(np.int64)
        pos = np.concatenate([np.arange(blk_off[r], blk_off[r] + prior[r]) for r in range(R)])
        poff = np.zeros(R + 1, np.int64)
        poff[1:] = np.cumsum(prior)
        ix.insert(keys[pos], poff, tbs.home[:R], bs.session[:R], 0)
        # timed: hash + match + route + insert, exactly the GPU step's work for n requests
        t0 = time.perf_counter()
        blk_off, keys = oracle.hash_blocks(toks, tok_off, W.BLOCK, W.DEFAULT_SEED)
        m = ix.match(keys, blk_off)
        tgt, br = oracle.route(m, bs.prompt_len[:R], bs.hist_len[:R], bs.turn[:R], bs.q, params, bs.rr_base)
        ix.insert(keys, blk_off, tgt, bs.session[:R], bs.epoch)
        dt = time.perf_counter() - t0
        return dt, keys, m, tgt, br

    cpus = os.sched_getaffinity(0)
    core = min(cpus)
    os.sched_setaffinity(0, {core})  # the oracle is single-threaded: one core, as taskset -c would
    try:
        dt, *_ = run(8)
        n = int(max(8, min(setup.args.n_req, 8 * budget_s / max(dt, 1e-6))))
        dt, keys, m, tgt, br = run(n)
    finally:
        os.sched_setaffinity(0, cpus)
    g_keys, g_m, g_t, g_b = gpu_out
    nk = len(keys)
    parity = (np.array_equal(g_keys[:nk], keys) and np.array_equal(g_m[:n], m) and np.array_equal(g_t[:n], tgt)
              and np.array_equal(g_b[:n], br))
    return dict(value=n / dt, unit="requests/s", cores=1, kind="oracle",
                sample=f"first {n} requests (of {setup.args.n_req}) of the last timed batch, hash+match+route+insert, "
                       f"start index restricted to their keys, single thread pinned to core {core}, {dt:.1f} s",
                cpu=host_cpu_model(), host_threads=os.cpu_count()), parity, n


def host_cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def measure_evict(setup):
    """LRU eviction of the whole start index (restored first), wall-clock with device syncs
    (the call ends in a stream sync of its own), exact count checked at full size (ceil(N f)
    entries go, status stays 0): first 5 % (the divergent-prefix configuration's rate),
    which leaves tombstones in place, then a third, which passes the tombstone limit and
    rebuilds the table (what every few 5 % evictions cost)."""
    import torch

    out = {}
    for name, (num, den) in (("in_place", (1, 20)), ("rebuild", (1, 3))):
        n0, _ = setup.index.stats()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        setup.index.evict(num, den)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        n1, st = setup.index.stats()
        out[name] = {"fraction": f"{num}/{den}", "ms": round(dt * 1e3, 2), "entries_before": n0,
                     "entries_after": n1, "entries_per_s": round(n0 / dt, 1),
                     "exact_count": bool(n0 - n1 == -(-n0 * num // den) and st == 0)}
    return out


def measure_variants(setup, b: int, reps: int = 20):
    """Route variants on the match rows of batch b (still in the output buffer), each
    event-timed over `reps` calls on the current stream."""
    import torch

    S, W, d, tb = setup.S, setup.W, setup.dev[b], setup.host[b]
    R, I = setup.matched.shape
    slack, n_run = setup.tw.decode_state(b)
    d_slack, d_run = torch.from_numpy(slack).cuda(), torch.from_numpy(n_run).cuda()
    tgt = torch.empty(R, dtype=torch.int32, device="cuda")
    br = torch.empty(R, dtype=torch.uint8, device="cuda")
    call = lambda: S.route_coloc(setup.matched, d["prompt_len"], d["hist_len"], d["turn"], d["q"], d_slack, d_run,
                                 W.DEFAULT_PARAMS, tb.batch.rr_base, target=tgt, branch=br)
    call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    alg = 4 * R * I + (8 + 8 + 4) * I + 12 * R + 5 * R  # c rows; q, slack, n_running; per-request in/out
    out = {"route_coloc": {"rule": "PD colocation (App. B): TPOT filter, LMetric score, no last resort",
                           "ms": round(ms, 4), "algorithmic_GBs": round(alg / ms / 1e6, 1),
                           "branches": np.bincount(br.cpu().numpy(), minlength=6).tolist()}}
    inputs = dict(route_coloc=(slack, n_run, tgt.cpu().numpy(), br.cpu().numpy(), b))
    # online load update: one wavefront routes the batch in order
    snap_t, _ = S.route(setup.matched, d["prompt_len"], d["hist_len"], d["turn"], d["q"], W.DEFAULT_PARAMS,
                        tb.batch.rr_base)
    snap_t = snap_t.cpu().numpy()
    q_out = torch.empty(I, dtype=torch.int64, device="cuda")
    ws = torch.empty(S.route_seq_ws_bytes(R), dtype=torch.uint8, device="cuda")
    call = lambda: S.route_seq(setup.matched, d["prompt_len"], d["hist_len"], d["turn"], d["q"], W.DEFAULT_PARAMS,
                               tb.batch.rr_base, target=tgt, branch=br, q_out=q_out, workspace=ws)
    call()
    seq_reps = max(2, reps // 4)
    e0.record()
    for _ in range(seq_reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / seq_reps
    st = tgt.cpu().numpy()
    out["route_seq"] = {"rule": "Sec. 4.2 rule, each request sees the queue updated by the earlier ones",
                        "ms": round(ms, 4), "requests_per_s": round(R / (ms / 1e3), 1),
                        "branches": np.bincount(br.cpu().numpy(), minlength=5).tolist(),
                        "targets_differing_from_batch_snapshot": int((st != snap_t).sum())}
    inputs["route_seq"] = (st, br.cpu().numpy(), q_out.cpu().numpy(), b)
    # the same rows as first turns: every decision is the sequential argmin over the
    # running loads (no stick, no last-resort shortcut)
    turn0 = torch.zeros_like(d["turn"])
    call = lambda: S.route_seq(setup.matched, d["prompt_len"], d["hist_len"], turn0, d["q"], W.DEFAULT_PARAMS,
                               tb.batch.rr_base, target=tgt, branch=br, q_out=q_out, workspace=ws)
    call()
    e0.record()
    for _ in range(seq_reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / seq_reps
    out["route_seq_all_scans"] = {"rule": "as route_seq, every request a first turn (each decision scans the "
                                          "running loads)",
                                  "ms": round(ms, 4), "requests_per_s": round(R / (ms / 1e3), 1),
                                  "branches": np.bincount(br.cpu().numpy(), minlength=5).tolist()}
    inputs["route_seq_all_scans"] = (tgt.cpu().numpy(), br.cpu().numpy(), q_out.cpu().numpy(), b)
    # the colocated rule, one request at a time: the queue and the request counts update
    n_out = torch.empty(I, dtype=torch.int64, device="cuda")
    ws = torch.empty(S.route_seq_coloc_ws_bytes(R, I), dtype=torch.uint8, device="cuda")
    call = lambda: S.route_seq_coloc(setup.matched, d["prompt_len"], d["hist_len"], d["turn"], d["q"], d_slack, d_run,
                                     W.DEFAULT_PARAMS, tb.batch.rr_base, target=tgt, branch=br, q_out=q_out,
                                     n_out=n_out, workspace=ws)
    call()
    e0.record()
    for _ in range(seq_reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / seq_reps
    sc = tgt.cpu().numpy()
    out["route_seq_coloc"] = {"rule": "PD colocation (App. B), each request sees the queue and request counts "
                                      "updated by the earlier ones",
                              "ms": round(ms, 4), "requests_per_s": round(R / (ms / 1e3), 1),
                              "branches": np.bincount(br.cpu().numpy(), minlength=6).tolist(),
                              "targets_differing_from_batch_snapshot": int((sc != inputs["route_coloc"][2]).sum())}
    inputs["route_seq_coloc"] = (sc, br.cpu().numpy(), q_out.cpu().numpy(), n_out.cpu().numpy(), b)
    # the Sec. 5.4 ablation's load-aware filter, load = queued prefill + 100 ms per running request
    load = d["q"] + d_run.to(torch.int64) * 100_000_000
    call = lambda: S.route_loadaware(setup.matched, d["prompt_len"], d["hist_len"], d["turn"], d["q"], load, (1, 2),
                                     W.DEFAULT_PARAMS, tb.batch.rr_base, target=tgt, branch=br)
    call()
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    la_t = tgt.cpu().numpy()
    out["route_loadaware"] = {"rule": "Sec. 5.4 ablation: stick unless prev's load > 1.5 x mean",
                              "ms": round(ms, 4), "branches": np.bincount(br.cpu().numpy(), minlength=5).tolist()}
    inputs["route_loadaware"] = (load.cpu().numpy(), la_t, br.cpu().numpy(), b)
    # the comparison scorers of the scoring template (Sec. 4.1, Sec. 5) on the same rows:
    # queued prefill in tokens (the queue's ns over C_LIN), load = requests running,
    # lam = 9/10 (a weight that favours reuse, as set for agentic workloads)
    q_tok = d["q"] // W.DEFAULT_PARAMS["c_lin"]
    B = W.DEFAULT_PARAMS["block_size"]
    lam = (9, 10)
    names = {S.SCORE_LOAD: "load_only", S.SCORE_TOKENS: "tokens_left_dynamo", S.SCORE_PRODUCT: "product_lmetric",
             S.SCORE_LINEAR: "weighted_sum", S.SCORE_HIT_FILTER: "hit_filter_preble"}
    sc_out, sc_in, sc_targets = {}, {}, {}
    for kind, name in names.items():
        call = lambda: S.route_score(kind, setup.matched, d["prompt_len"], q_tok, d_run, B, lam, tb.batch.rr_base,
                                     target=tgt, branch=br)
        call()
        e0.record()
        for _ in range(reps):
            call()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        st, sb = tgt.cpu().numpy(), br.cpu().numpy()
        sc_out[name] = {"ms": round(ms, 4), "same_target_as_smetric_batch": int((st == snap_t).sum()),
                        "hit_filter_decisions": int((sb == 7).sum())}
        sc_in[kind] = (st, sb)
        sc_targets[name] = st
    out["route_score"] = {"rule": "Sec. 4.1 scoring template: argmin of a comparison scorer, lam = 9/10",
                          "scorers": sc_out}
    inputs["route_score"] = (q_tok.cpu().numpy(), lam, sc_in, b)
    # load imbalance (Sec. 4.1) of the batch-snapshot and the load-aware decisions: arrivals
    # spread over 10 min, each request running 20 s, 30 s windows
    rng = np.random.default_rng(b)
    t0 = np.sort(rng.integers(0, 600_000, R)).astype(np.int64)
    d_t0 = torch.from_numpy(t0).cuda()
    d_t1 = d_t0 + 20_000
    imb = {}
    for name, tg in (("smetric_batch", snap_t), ("loadaware", la_t), *sc_targets.items()):
        gs, gm, _ = S.imbalance(torch.from_numpy(tg.astype(np.int32)).cuda(), d_t0, d_t1, I, 30_000, 21)
        gs, gm = gs.cpu().numpy(), gm.cpu().numpy()
        ratio = gm * I / np.maximum(gs, 1)
        imb[name] = {"median": round(float(np.median(ratio[gs > 0])), 3), "max": round(float(ratio.max()), 3)}
    out["imbalance_30s_windows"] = imb
    # session reconstruction from block hashes on a multi-session trace
    tr = W.session_trace(n_users=1024, sessions_per_user=4, turns=8)
    blk_off, nb = S.block_offsets(tr.tok_off)
    d_tok, d_toff, d_boff = (torch.from_numpy(tr.tokens).cuda(), torch.from_numpy(tr.tok_off).cuda(),
                             torch.from_numpy(blk_off).cuda())
    d_user, d_turn = torch.from_numpy(tr.user).cuda(), torch.from_numpy(tr.turn).cuda()
    keys = S.hash_blocks(d_tok, d_toff, d_boff, nb)
    par = torch.empty(tr.n_req, dtype=torch.int32, device="cuda")
    ses = torch.empty(tr.n_req, dtype=torch.int32, device="cuda")
    ws = torch.empty(S.sessions_ws_bytes(tr.n_req), dtype=torch.uint8, device="cuda")
    call = lambda: S.sessions(keys, d_boff, nb, d_user, d_turn, parent=par, session=ses, workspace=ws)
    call()
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    gp, gs = par.cpu().numpy(), ses.cpu().numpy()
    keep = ~tr.compacted
    out["sessions"] = {"rule": "App. A: follow-up = same user, turn + 1, block-hash prefix",
                       "trace": f"{len(np.unique(tr.user))} users x 4 sessions x 8 turns, {tr.n_req} requests, "
                                f"{nb} blocks, 5% compactions, 3% retries",
                       "ms": round(ms, 4), "requests_per_s": round(tr.n_req / (ms / 1e3), 1),
                       "blocks_per_s": round(nb / (ms / 1e3), 1), "linked": int((gp >= 0).sum()),
                       "sessions_found": int(len(np.unique(gs))), "true_sessions": int(len(np.unique(tr.true_session))),
                       "parent_agreement_excluding_compactions": round(float((gp[keep] == tr.true_parent[keep]).mean()), 6)}
    inputs["sessions"] = (tr, blk_off, gp, gs)
    return out, inputs


def variants_parity(setup, inputs) -> dict:
    """The variants' whole-batch outputs against the oracle (CPU-baseline leg only)."""
    import oracle

    slack, n_run, gt, gb, b = inputs["route_coloc"]
    bt = setup.host[b].batch
    ot, ob = oracle.route_coloc(setup.matched.cpu().numpy(), bt.prompt_len, bt.hist_len, bt.turn, bt.q, slack, n_run,
                                setup.W.DEFAULT_PARAMS, bt.rr_base)
    res = {"route_coloc": {"requests": int(len(ot)), "bit_exact": bool(np.array_equal(ot, gt) and np.array_equal(ob, gb))}}
    gt, gb, gq, b = inputs["route_seq"]
    bt = setup.host[b].batch
    ot, ob, oq = oracle.route_seq(setup.matched.cpu().numpy(), bt.prompt_len, bt.hist_len, bt.turn, bt.q,
                                  setup.W.DEFAULT_PARAMS, bt.rr_base)
    res["route_seq"] = {"requests": int(len(ot)), "bit_exact": bool(np.array_equal(ot, gt) and np.array_equal(ob, gb)
                                                                    and np.array_equal(oq, gq))}
    gt, gb, gq, b = inputs["route_seq_all_scans"]
    ot, ob, oq = oracle.route_seq(setup.matched.cpu().numpy(), bt.prompt_len, bt.hist_len, np.zeros_like(bt.turn),
                                  bt.q, setup.W.DEFAULT_PARAMS, bt.rr_base)
    res["route_seq_all_scans"] = {"requests": int(len(ot)), "bit_exact": bool(
        np.array_equal(ot, gt) and np.array_equal(ob, gb) and np.array_equal(oq, gq))}
    gt, gb, gq, gn, b = inputs["route_seq_coloc"]
    bt = setup.host[b].batch
    slack, n_run = inputs["route_coloc"][0], inputs["route_coloc"][1]
    ot, ob, oq, on = oracle.route_seq_coloc(setup.matched.cpu().numpy(), bt.prompt_len, bt.hist_len, bt.turn, bt.q,
                                            slack, n_run, setup.W.DEFAULT_PARAMS, bt.rr_base)
    res["route_seq_coloc"] = {"requests": int(len(ot)), "bit_exact": bool(
        np.array_equal(ot, gt) and np.array_equal(ob, gb) and np.array_equal(oq, gq) and np.array_equal(on, gn))}
    load, gt, gb, b = inputs["route_loadaware"]
    bt = setup.host[b].batch
    ot, ob = oracle.route_loadaware(setup.matched.cpu().numpy(), bt.prompt_len, bt.hist_len, bt.turn, bt.q, load,
                                    (1, 2), setup.W.DEFAULT_PARAMS, bt.rr_base)
    res["route_loadaware"] = {"requests": int(len(ot)), "bit_exact": bool(np.array_equal(ot, gt) and np.array_equal(ob, gb))}
    q_tok, lam, sc_in, b = inputs["route_score"]
    bt = setup.host[b].batch
    n_run = inputs["route_coloc"][1]
    m = setup.matched.cpu().numpy()
    exact = True
    for kind, (gt, gb) in sc_in.items():
        ot, ob = oracle.route_score(kind, m, bt.prompt_len, q_tok, n_run, setup.W.DEFAULT_PARAMS["block_size"], lam,
                                    bt.rr_base)
        exact = exact and bool(np.array_equal(ot, gt) and np.array_equal(ob, gb))
    res["route_score"] = {"requests": int(len(bt.prompt_len)), "scorers": len(sc_in), "bit_exact": exact}
    tr, blk_off, gp, gs = inputs["sessions"]
    ob, ok = oracle.hash_blocks(tr.tokens, tr.tok_off, setup.W.BLOCK, setup.W.DEFAULT_SEED)
    op, os_ = oracle.sessions(ok, ob, tr.user, tr.turn)
    res["sessions"] = {"requests": int(tr.n_req), "bit_exact": bool(np.array_equal(op, gp) and np.array_equal(os_, gs))}
    return res


COPY_BYTES = 1 << 30


def insert_checks(setup, b: int, keys_h, matched_h, target_h, n_after: int) -> dict:
    """Full-size checks of batch b's post-route insert into the start index (untimed).
    (i) Append-only (Sec. 2; the target caches the prompt it prefills, Sec. 4.2): matching
        the batch again gives matched[r][target[r]] = its block count for every request.
    (ii) The entry count grows by exactly the distinct pairs (key_j, target_r) with
        j >= matched[r][target_r]: the start index is prefix-closed on every instance (whole
        prior turns; filler keys match nothing), so the target holds none of those blocks
        and all the others; nothing is evicted."""
    torch = setup.torch
    d = setup.dev[b]
    off = d["blk_off_h"]
    nb = np.diff(off)
    R = len(nb)
    c_t = matched_h[np.arange(R), target_h].astype(np.int64)
    starts, cnt = off[:-1] + c_t, nb - c_t
    base = np.concatenate([[0], np.cumsum(cnt)[:-1]])
    pos = np.repeat(starts - base, cnt) + np.arange(int(cnt.sum()))
    k = keys_h[pos]
    t = np.repeat(target_h.astype(np.uint64), cnt)
    order = np.lexsort((t, k))
    ks, ts = k[order], t[order]
    expect = int(len(ks) > 0) + int(np.count_nonzero((ks[1:] != ks[:-1]) | (ts[1:] != ts[:-1])))
    got = n_after - setup.start_entries
    m2 = torch.empty_like(setup.matched)
    setup.path_only(b, 1, m2)
    m2 = m2.cpu().numpy()
    whole = m2[np.arange(R), target_h] == nb
    return {"append_only_all_requests": bool(whole.all()), "requests": int(R),
            "requests_failing": int((~whole).sum()),
            "new_entries": {"got": int(got), "expected_distinct_new_pairs": expect, "equal": bool(got == expect)}}


def main():
    args = parse()
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, args.steps))
        return
    if args.summarize_sq:
        print(summarize_sq(args.summarize_sq[0], args.steps, args.summarize_sq[1]))
        return
    if args.summarize_pmc:
        res, md = summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.steps, COPY_BYTES,
                                args.summarize_pmc[2])
        with open(args.traffic, "w") as f:
            json.dump(res, f, indent=1)
        print(md)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: the matching/routing path is "
                                   "not sharded across GPUs (pass --gpus 1)"}))
        sys.exit(2)
    import torch

    torch.cuda.set_device(0)
    setup = Setup(args)
    S = setup.S
    # warm-up (untimed), each step from the start index
    for i in range(args.warmup):
        setup.restore()
        setup.step(setup.batch_of(i))
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    wall = 0.0
    for k in range(args.steps):
        setup.restore()  # untimed: every step starts from the same index
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        setup.step(setup.batch_of(args.warmup + k), evs[k])
        torch.cuda.synchronize()
        wall += time.perf_counter() - t0
    per = {n: float(np.mean([evs[k][i].elapsed_time(evs[k][i + 1]) for k in range(args.steps)]))
           for i, n in enumerate(Setup.CALLS)}
    n_after, st = setup.index.stats()
    assert st == 0, f"index status {st}"
    # the last timed batch, checked at full size (untimed)
    last = setup.batch_of(args.warmup + args.steps - 1)
    nb_last = setup.dev[last]["n_blocks"]
    gpu_out = (setup.keys[:nb_last].cpu().numpy(), setup.matched.cpu().numpy(), setup.target.cpu().numpy(),
               setup.branch.cpu().numpy())
    n_probed, n_search = (None, None) if args.direct else setup.index.probe_stats(setup.probe_state, nb_last)
    checks = insert_checks(setup, last, gpu_out[0], gpu_out[1], gpu_out[2], n_after)
    alg = algorithmic_bytes(setup, last, gpu_out[1], args.n_inst, n_probed, n_search)
    R = args.n_req
    tokens = float(np.mean([setup.host[setup.batch_of(args.warmup + k)].batch.n_tokens for k in range(args.steps)]))
    ms_step = wall * 1e3 / args.steps
    probe_match_ms = per["probe"] + per["match"]
    gbs = {"hash": alg["hash"] / per["hash"] / 1e6}
    if args.direct:
        gbs["match"] = alg["match"] / per["match"] / 1e6
    else:
        gbs["probe"] = alg["probe"] / per["probe"] / 1e6
        gbs["match"] = alg["match_scan"] / per["match"] / 1e6
    dominant = max(("hash", "probe", "match", "route"), key=lambda k: per[k])
    cfg = {"workload": f"throughput: {args.n_inst} instances, {R} requests/batch, lognormal(24576, 0.6) prompts in "
                       f"[1024, 131072], 70% prior-turn blocks, 64 Zipf(1.2) 4096-token prefixes; start index "
                       f"{setup.start_entries} entries in {setup.index.n_slots} slots (restored before every step)",
           "n_instances": args.n_inst, "requests_per_batch": R, "block_size": 16,
           "index_entries_start": setup.start_entries, "index_prior_turn_entries": setup.prior_entries,
           "index_slots": setup.index.n_slots,
           "occupancy_start": round(setup.start_entries / setup.index.n_slots, 4),
           "index_entries_after_step": n_after, "index_capacity": setup.capacity,
           "distinct_batches": setup.n_distinct, "tokens_per_batch": int(tokens)}
    tr = {}
    if os.path.exists(args.traffic) and not args.direct:
        t = json.load(open(args.traffic))
        # counters of the current kernels on this workload only
        if t.get("sources_sha256_16") == kernel_sources_hash() and t.get("workload") == workload_key(cfg):
            tr = t
    launches = (lambda c: None if args.direct else CALL_KERNELS[c])
    show = (lambda c: c) if args.direct else (lambda c: Setup.SHOW[c])
    roof = {"bound": "hbm", "kernel": show(dominant), "launches": launches(dominant),
            "achieved": round(gbs.get(dominant, 0.0), 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs.get(dominant, 0.0) / HBM_PEAK_GBS, 4),
            "traffic": round(tr[dominant]) if dominant in tr else None}
    if dominant == "probe" and not args.direct:
        roof["per_launch"] = {"blocks": alg["blocks"], "blocks_probed": alg["blocks_probed"],
                              "bound_search_probes": alg["search_probes"], "bytes_per_probe": 72,
                              "necessary_probes": alg["probes"],
                              "necessary_fraction_of_blocks": round(alg["probes"] / max(alg["blocks"], 1), 4),
                              "descriptor_bytes_written": alg["descriptor"]}
    # the post-route insert: one bucket burst per pair, 16 B per new entry, 8 B per refresh
    new_pairs = n_after - setup.start_entries
    n_blk = alg["blocks"]
    ins_b = 64 * n_blk + 16 * new_pairs + 8 * (n_blk - new_pairs)
    ins_gbs = ins_b / per["insert"] / 1e6
    insert = {"kernel": "insert", "launches": launches("insert"), "new_pairs": int(new_pairs),
              "achieved": round(ins_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
              "frac": round(ins_gbs / HBM_PEAK_GBS, 4), "traffic": round(tr["insert"]) if "insert" in tr else None}
    path_bytes = alg["hash"] + alg["match"]
    path_ms = per["hash"] + probe_match_ms
    path_gbs = path_bytes / path_ms / 1e6
    path_gbs_noh = (path_bytes - alg["H"]) / path_ms / 1e6
    out = {
        "metric": METRIC, "value": round(R / (ms_step / 1e3), 1), "unit": "requests/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": cfg,
        "path": ("direct" if args.direct else "hash + region partition in one call, then the region-ordered lookup")
                + "; one batch at a time, the index restored (untimed) before every step",
        "prompt_tokens_matched_per_s": round(tokens / ((per["hash"] + probe_match_ms) / 1e3), 1),
        # the decision alone (hash, lookup, match, route: the insert follows it), by event time
        "requests_routed_per_s_before_insert": round(R / ((per["hash"] + probe_match_ms + per["route"]) / 1e3), 1),
        "kernel_ms": {show(k): round(per[k], 4) for k in Setup.CALLS if not (args.direct and k == "probe")},
        "algorithmic_GBs": {show(k): round(v, 1) for k, v in gbs.items()},
        "hash_probe_path": {"GBs": round(path_gbs, 1), "frac_of_peak": round(path_gbs / HBM_PEAK_GBS, 4),
                            "frac_of_peak_without_shared_prefix_bitmaps": round(path_gbs_noh / HBM_PEAK_GBS, 4),
                            "bytes": path_bytes, "shared_prefix_bitmap_bytes": alg["H"],
                            "necessary_probes": alg["probes"], "blocks": alg["blocks"]},
        "roofline": roof,
        "roofline_insert": insert,
        "branches": {"counts": np.bincount(gpu_out[3], minlength=5).tolist(),
                     "names": ["first-turn", "evicted", "stick", "last-resort", "migrate"]},
        "insert_checks": checks,
    }
    if args.overlap_path and not args.direct:  # batch k+1's hash beside batch k's lookup and match
        setup.restore()
        m2 = [torch.empty_like(setup.matched), torch.empty_like(setup.matched)]
        batches = [setup.batch_of(args.warmup + k) for k in range(args.steps)]
        setup.path_overlapped(batches[:2], m2)  # warm
        dt = setup.path_overlapped(batches, m2)
        ms = dt * 1e3 / len(batches)
        out["hash_probe_path_overlapped"] = {
            "ms_per_batch": round(ms, 4), "GBs": round(path_bytes / ms / 1e6, 1),
            "frac_of_peak": round(path_bytes / ms / 1e6 / HBM_PEAK_GBS, 4),
            "how": "two streams: the next batch's hash + partition beside this batch's lookup + match; "
                   "wall time over the timed batches"}
        del m2
    if args.overlap_step and not args.direct:  # batch k+1's hash beside batch k's lookup .. insert
        setup.restore()
        batches = [setup.batch_of(args.warmup + k) for k in range(args.steps)]
        setup.step_overlapped(batches[:2])  # warm
        dt = setup.step_overlapped(batches)
        ms = dt * 1e3 / len(batches)
        out["step_overlapped"] = {
            "ms_per_step": round(ms, 4), "requests_per_s": round(R / (ms / 1e3), 1),
            "how": "two streams: the next batch's hash + partition beside this batch's lookup, match, route and "
                   "insert; the index restored between steps (untimed, after both streams finished); wall time "
                   "over the timed batches, the first batch's hash included"}
        setup.restore()
    if args.calibrate_copy:  # a device copy of known size, for the HBM counters' scale
        src = torch.ones(COPY_BYTES, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    variants, var_inputs = measure_variants(setup, last)
    out["variants"] = variants
    setup.restore()
    out["evict"] = measure_evict(setup)
    if not args.no_cpu_baseline:
        cb, parity, n_s = cpu_baseline(setup, last, args.cpu_seconds, gpu_out)
        out["cpu_baseline"] = cb
        out["sampled_parity"] = {"batch": "last timed", "requests": n_s, "bit_exact": bool(parity)}
        out["sampled_parity"]["variants"] = variants_parity(setup, var_inputs)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
