#!/usr/bin/env python3
"""Benchmark of the NLB forward-recent-sampling hot path on one MI355X.

A step is one batch of the stream through the whole hot path, in the
paper's order (Sec. 4.2): nlb_sample answers the batch's queries (both
endpoints and one negative per link, at the link's time) from the current
tables, then nlb_insert_batch applies the batch's links.  Inputs (the whole
stream in the batch-blocked layout, feature tables, time parameters) are
resident in HBM before timing starts; the tables are first filled by
inserting the stream up to the start batch.

Prints one JSON line.  `value` is links per second through the whole step;
queries/s and the kernel-only rates are extra fields.  `roofline` reports
the sample call (the dominant work: sample_gather, plus tenc_stream on
large launches) against MI355X peak HBM bandwidth, timed with HIP events on
the stream the kernels run on.  `cpu_baseline` times the CPU oracle on the
GPU machine's host: its insertion over the stream up to the GPU's timed window,
then retrieval and insertion on the window's first batches.  `streamed`
repeats the step with the batches arriving from host memory (pinned
buffers, copied to the device on a second stream, ordered by events), once
from a live host generator and once from batches staged beforehand.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
# Batches whose time encoding is at least this large run it on a second
# stream (nlb_time_encode) beside the insert (and status update); smaller
# ones keep nlb_sample's one-stream form.
ENCODE_STREAM_MIN_BYTES = 1 << 30


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", type=int, default=5)
    ap.add_argument("--start-batch", type=int, default=None,
                    help="first batch of the warmup (default: the middle of the stream)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--hop2", action="store_true",
                    help="also answer every step's second hop (Sec. 4.4) with nlb_sample_hop2, "
                         "ids only, and report it separately")
    ap.add_argument("--aggregate", action="store_true",
                    help="retrieve with the fused eq. (4) attention aggregation (nlb_aggregate, "
                         "random weights) instead of nlb_sample, and report that kernel")
    ap.add_argument("--heads", type=int, default=1,
                    help="attention heads of --aggregate (App. E uses two)")
    ap.add_argument("--rnn", action="store_true",
                    help="also update the node statuses after every batch (Sec. 4.4 GRU, "
                         "nlb_rnn_update, random weights): the node-feature rows when the workload "
                         "has them, else an fp32 status table of width 100")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="before the benchmark, run a plain elementwise copy of this many MiB "
                         "five times (a known-traffic kernel for calibrating HBM counters)")
    ap.add_argument("--gather-probe-mb", type=int, default=0,
                    help="before the benchmark, gather this many MiB of 256-byte rows, each "
                         "row once, from a random permutation of a table 8x larger, five times "
                         "(a known-traffic random gather for calibrating HBM counters)")
    ap.add_argument("--graph", action="store_true",
                    help="capture the K timed steps (each batch's sample, insert and, with --rnn, "
                         "status update, at their own stream offsets) in one HIP graph and time one "
                         "replay of it: the step without host launch costs")
    ap.add_argument("--serial-encode", action="store_true",
                    help="compute each retrieval's time encoding inside nlb_sample on the one "
                         "stream, instead of with nlb_time_encode on a second stream beside the "
                         "insert (and status update) that follow")
    ap.add_argument("--encode-stream", action="store_true",
                    help="use the second stream for the time encoding also when a batch's "
                         "encoding is under 1 GiB or with --hop2 (by default such steps keep "
                         "the one-stream form: for small batches the extra launch and events cost "
                         "more than the overlap saves, and the second hop's table reads and the "
                         "encoding slow each other down)")
    ap.add_argument("--encode-depth", type=int, default=1,
                    help="sets of retrieval output buffers the steps take turns over: with 2, a "
                         "batch's time encoding also runs beside the next batch's table reads")
    ap.add_argument("--streamed-steps", type=int, default=500,
                    help="steps of the host-streamed legs (0: skip them)")
    ap.add_argument("--cpu-plan", action="store_true",
                    help="no GPU work: time the CPU oracle over the whole stream (every insert) and "
                         "retrieval on the batches 0-9, every 1000th and the last 10, and print "
                         "that as the JSON line")
    return ap.parse_args()


def sample_bytes(w, valid_slots, queries):
    """Algorithmic HBM bytes of one sample launch: what the method must move.
    Reads: node id + query time (8 B), the s table slots (12 B each), the
    link-feature and neighbour rows of valid slots and the self row.
    Writes: nbr/eid/ts (12 B per slot), the fp32 time encoding (4*d_time per
    slot), feature rows of every slot (zeros when invalid) and the self row."""
    s, erb, nrb = w.s, w.row_bytes("edge"), w.row_bytes("node")
    reads = queries * (8 + 12 * s + nrb) + valid_slots * (erb + nrb)
    writes = queries * s * (12 + 4 * w.d_time + erb + nrb) + queries * nrb
    return reads + writes


# Per call: the summary file (by workload name) and the sources its kernels
# are built from.
COUNTER_SOURCES = {
    "nlb_sample": ("sample_gather_{}.md", ("nlb.hip", "nlb_internal.h", "nlb_divide.h")),
    "nlb_aggregate": ("aggregate_packed_{}.md",
                      ("aggregate.hip", "nlb_internal.h", "nlb_pieces.h", "nlb_divide.h")),
}


def kernel_source_hash(call="nlb_sample"):
    """sha256 over the sources of a call's kernels, the key under which
    counter summaries stay valid."""
    import hashlib
    hs = hashlib.sha256()
    for f in COUNTER_SOURCES[call][1]:
        hs.update(open(os.path.join(ROOT, "paper_2402_01964_amd", "csrc", f), "rb").read())
    return hs.hexdigest()


def measured_traffic(w, call="nlb_sample"):
    """HBM bytes per call (all its launches) from the committed rocprofv3
    counter summary of this workload, or None when there is none or the
    kernel sources have changed since the counters were taken."""
    import re
    path = os.path.join(ROOT, "profiles", COUNTER_SOURCES[call][0].format(w.name))
    if not os.path.exists(path):
        return None
    m = re.search(r"counters: workload=(\S+) call=(\S+) traffic_bytes_per_call=(\S+) "
                  r"kernel_source_sha256=([0-9a-f]+)", open(path).read())
    if not m or m.group(1) != w.name or m.group(2) != call:
        return None
    if kernel_source_hash(call) != m.group(4):
        return None
    return float(m.group(3))


def aggregate_kernel(w, queries, cus, heads=1):
    """The eq. (4) kernel a launch of `queries` takes on this workload's
    shapes (the library's own choice, restated for the record): with one or
    two heads, the packed form for tables of at most 16 slots when its query
    groups hold at least 8 queries, else the per-query form; more heads take
    the tiled form."""
    if heads > 2:
        return "aggregate_fused"
    gq = min(16, max(1, -(-queries // (cus * 8))))
    return "aggregate_packed" if w.s <= 16 and gq >= 8 else "aggregate_rows"


def hop2_bytes(w, hop1_valid, queries):
    """Algorithmic bytes of one ids-only second-hop launch over `queries`
    first-hop queries: per first-hop entry its neighbour id and the query
    time (8 B) and, when valid, the neighbour's s slots (12 B each); writes
    nbr/eid/ts for s*s slots per query (12 B each)."""
    return queries * w.s * 8 + hop1_valid * 12 * w.s + queries * w.s * w.s * 12


PEAK_BF16_TFLOPS = 2500.0


def aggregate_flops(w, valid_slots, queries, hidden=64, heads=1):
    """Algorithmic matrix FLOPs of eq. (4) as computed (no padding, one
    product per weight): MLP_in's first layer and each head's attention
    logit for every valid slot; MLP_in's second layer, which is affine, once
    on each query's softmax-weighted sums (each head's slice of its outputs),
    and MLP_out's two layers, for every query.  (Applying the second layer to
    every slot, in the order the equation is written, would add 2 H^2 per
    valid slot.)"""
    d_in = w.node_dim + w.edge_dim + w.d_time
    per_slot = 2 * (d_in * hidden + heads * hidden)
    per_query = 2 * (hidden * hidden + (w.node_dim + hidden) * hidden + hidden * hidden)
    return valid_slots * per_slot + queries * per_query


def aggregate_bytes(w, valid_slots, queries, hidden=64):
    """Algorithmic HBM bytes of one aggregation launch: query ids and times,
    the table slots, the rows of valid slots and the self row; Z written."""
    erb, nrb = w.row_bytes("edge"), w.row_bytes("node")
    return queries * (8 + 12 * w.s + nrb + 4 * hidden) + valid_slots * (erb + nrb)


def rnn_flops(w, d, winners):
    """Algorithmic matrix FLOPs of one status update: for each node updated
    (the winners: distinct endpoints of the batch), the GRU's input and
    hidden products, 2 * 3d * (d + d_time + edge_dim) + 2 * 3d * d."""
    return winners * 2 * 3 * d * (2 * d + w.d_time + w.edge_dim)


def rnn_bytes(w, d, status_bytes, links, winners):
    """Algorithmic HBM bytes of one status update: link ids and times; per
    winner its own and its partner's status row and its link row read, and
    its new row written."""
    srb = d * status_bytes
    return links * 12 + winners * (3 * srb + w.row_bytes("edge"))


def binding_roofline(flops, nbytes, seconds):
    """The roofline that bounds a kernel doing `flops` matrix FLOPs (bf16)
    and moving `nbytes` algorithmic HBM bytes: the one whose peak needs the
    longer time (HBM when nbytes / 8 TB/s exceeds flops / 2.5 PFLOP/s), with
    the achieved rate against it; the other is reported beside it."""
    t_hbm = nbytes / (PEAK_HBM_GBPS * 1e9)
    t_mfma = flops / (PEAK_BF16_TFLOPS * 1e12)
    hbm = {"achieved": nbytes / seconds / 1e9, "peak": PEAK_HBM_GBPS, "unit": "GB/s"}
    mfma = {"achieved": flops / seconds / 1e12, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"}
    for d in (hbm, mfma):
        d["frac"] = d["achieved"] / d["peak"]
    bound, main, other = ("hbm", hbm, mfma) if t_hbm >= t_mfma else ("mfma", mfma, hbm)
    return dict(bound=bound, **main, other={"bound": "mfma" if bound == "hbm" else "hbm", **other},
                floor_seconds=max(t_hbm, t_mfma))


def insert_bytes(links):
    """Algorithmic bytes of one insert: 12 B of input per link, and per
    offer an 8 B key read-modify-write plus a 4 B neighbour write."""
    return links * (12 + 2 * (8 + 8 + 4))


def host_info():
    """The host the CPU figures come from: CPU model, logical CPUs, and the
    CPUs this process may run on."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        allowed = len(os.sched_getaffinity(0))
    except AttributeError:
        allowed = os.cpu_count()
    return {"cpu_model": model, "nproc": os.cpu_count(), "cpus_allowed": allowed}


class _HostRows:
    """Full-size host feature tables for the oracle, rows generated on first
    use (untouched rows stay unmaterialised zero pages)."""

    def __init__(self, w, links_upto):
        import numpy as np
        self.w, self.ef, self.nf = w, None, None
        if w.edge_dim:
            self.ef = np.zeros((links_upto, w.edge_dim), np.float32 if w.elem_bytes("edge") == 4 else np.uint16)
            self.e_done = np.zeros(links_upto, bool)
        if w.node_dim:
            self.nf = np.zeros((w.num_nodes, w.node_dim), np.float32 if w.elem_bytes("node") == 4 else np.uint16)
            self.n_done = np.zeros(w.num_nodes, bool)

    def need(self, o, q):
        """Materialise the rows a retrieval of queries q will read."""
        import numpy as np

        import synth
        nbr, _, eid = o.export_nodes(q)
        if self.nf is not None:
            rows = np.unique(np.concatenate([q, nbr[nbr >= 0]]))
            rows = rows[~self.n_done[rows]]
            if len(rows):
                self.nf[rows] = synth.host_feature_rows(self.w, "node", rows)
                self.n_done[rows] = True
        if self.ef is not None:
            rows = np.unique(eid[eid != 0xFFFFFFFF]).astype(np.int64)
            rows = rows[rows < len(self.ef)]
            rows = rows[~self.e_done[rows]]
            if len(rows):
                self.ef[rows] = synth.host_feature_rows(self.w, "edge", rows)
                self.e_done[rows] = True


def _stream_batches(w, b0, b1):
    """Host batches b0 .. b1-1 as (b, src, dst, t, neg), generated in chunks."""
    import synth
    if not w.stateless:
        whole = synth.host_links(w)
        for b in range(b0, b1):
            lo, hi = w.batch_range(b)
            yield (b, *(x[lo:hi] for x in whole))
        return
    per = max(1, 20_000_000 // w.batch)
    for c0 in range(b0, b1, per):
        c1 = min(b1, c0 + per)
        lo, hi = w.batch_range(c0)[0], w.batch_range(c1 - 1)[1]
        src, dst, t, neg = synth.host_links(w, lo, hi)
        for b in range(c0, c1):
            a, z = w.batch_range(b)
            yield b, src[a - lo:z - lo], dst[a - lo:z - lo], t[a - lo:z - lo], neg[a - lo:z - lo]


def cpu_baseline(w, first, budget_s, agg_weights=None, hop2=False, heads=1):
    """The CPU oracle, one thread, on the GPU machine's host.  Insertion is
    timed over every link of batches 0 .. first-1 (the replay that brings the
    oracle to the GPU's timed window); then, from batch `first` on, each
    batch's retrieval (sample -- or, with agg_weights, the eq. (4)
    aggregation; with hop2 also the second hop's ids) and its insertion are
    timed separately until the retrieval budget is used.  Stream generation
    and feature-row generation are outside the timed regions."""
    import numpy as np

    import oracle
    import synth
    o = oracle.Oracle(w.num_nodes, w.s, w.alpha, w.table_seed)
    fw, fb = synth.time_params(w)
    ins_s = 0.0
    ins_links = 0
    for b, src, dst, t, _ in _stream_batches(w, 0, first):
        t0 = time.perf_counter()
        o.insert(src, dst, t)
        ins_s += time.perf_counter() - t0
        ins_links += len(src)
    rows = _HostRows(w, w.links)
    q_s = win_ins_s = 0.0
    queries = win_links = 0
    b_end = first
    for b, src, dst, t, neg in _stream_batches(w, first, w.batches):
        if q_s >= budget_s:
            break
        q = np.concatenate([src, dst, neg])
        tq = np.concatenate([t, t, t])
        rows.need(o, q)
        t0 = time.perf_counter()
        if agg_weights is not None:
            o.aggregate(q, tq, fw, fb, rows.ef, rows.nf, agg_weights, heads=heads)
        else:
            r1 = o.sample(q, tq, fw, fb, rows.ef, rows.nf)
            if hop2:
                o.sample_hop2(r1["nbr"], tq, want=("nbr", "eid", "ts"))
        t1 = time.perf_counter()
        o.insert(src, dst, t)
        t2 = time.perf_counter()
        q_s += t1 - t0
        win_ins_s += t2 - t1
        queries += len(q)
        win_links += len(src)
        b_end = b + 1
    ins_rate = (ins_links + win_links) / (ins_s + win_ins_s)
    q_rate = queries / q_s
    what = "aggregate (eq. (4))" if agg_weights is not None else "sample, second hop" if hop2 else "sample"
    return {"value": win_links / (q_s + win_ins_s), "unit": "links/s", "cores": 1, "kind": "oracle",
            "queries_per_s": q_rate, "insert_links_per_s": ins_rate,
            "insert_window_links_per_s": win_links / win_ins_s,
            "seconds": ins_s + q_s + win_ins_s, "host": host_info(),
            "sample": f"one thread; insertion timed over batches 0..{b_end - 1} ({ins_links + win_links} links); "
                      f"{what} then insert timed on batches {first}..{b_end - 1} ({queries} queries, "
                      f"{win_links} links), the GPU's timed window; value = links/s through those "
                      f"steps"}


def cpu_plan(w):
    """The CPU oracle over the whole stream, one thread: every insertion
    timed, and retrieval (every query, all outputs) timed on the batches
    0-9, every 1000th and the last 10.  The retrieval rate of those batches
    is extrapolated to the whole stream (labelled as such)."""
    import numpy as np

    import oracle
    import synth
    nb = w.batches
    chosen = sorted(set(range(min(10, nb))) | set(range(0, nb, 1000)) | set(range(max(0, nb - 10), nb)))
    o = oracle.Oracle(w.num_nodes, w.s, w.alpha, w.table_seed)
    fw, fb = synth.time_params(w)
    rows = _HostRows(w, w.links)
    ins_s = q_s = 0.0
    queries = 0
    t_start = time.perf_counter()
    for b, src, dst, t, neg in _stream_batches(w, 0, nb):
        if b in chosen:
            q = np.concatenate([src, dst, neg])
            tq = np.concatenate([t, t, t])
            rows.need(o, q)
            t0 = time.perf_counter()
            o.sample(q, tq, fw, fb, rows.ef, rows.nf)
            q_s += time.perf_counter() - t0
            queries += len(q)
        t0 = time.perf_counter()
        o.insert(src, dst, t)
        ins_s += time.perf_counter() - t0
        if b % 1000 == 999:
            print(f"bench: oracle plan at batch {b + 1}", file=sys.stderr, flush=True)
    q_rate = queries / q_s
    all_q = 3 * w.links
    return {"metric": "CPU oracle: interactions/s inserted, queries/s sampled", "workload": w.name,
            "insert_links_per_s": w.links / ins_s, "insert_seconds": ins_s, "links": w.links,
            "sample_queries_per_s": q_rate, "sample_seconds": q_s, "sampled_queries": queries,
            "sampled_batches": len(chosen),
            "extrapolated_full_stream_sample_seconds": all_q / q_rate,
            "extrapolated_links_per_s_through_steps": w.links / (ins_s + all_q / q_rate),
            "extrapolation": "sample time of all 3 x links queries extrapolated from the timed "
                             "batches' per-query rate",
            "cores": 1, "kind": "oracle", "host": host_info(),
            "wall_seconds": time.perf_counter() - t_start}


class EncodeStream:
    """The time encoding of each retrieval on a second stream.  The table
    reads (nlb_sample without its tenc output) stay on the current stream;
    nlb_time_encode runs on this stream after them, beside what follows on
    the current stream (the encoding reads only the timestamp output and the
    query times).  Retrievals take turns over ``depth`` sets of output
    buffers: join() makes the current stream wait for the encoding that last
    used the set the next retrieval will write, so with two sets a batch's
    encoding also runs beside the next batch's table reads."""

    def __init__(self, dev, depth=1):
        import torch
        self.stream = torch.cuda.Stream(device=dev)
        self.depth = depth
        self.gathered = torch.cuda.Event()
        self.encoded = [torch.cuda.Event() for _ in range(depth)]
        self.used = [None] * depth    # the event that marks each set's last encoding
        self.count = 0

    @property
    def slot(self):
        """The output set the next retrieval writes."""
        return self.count % self.depth

    def sample_into(self, table, q, tq, o, events=None):
        """``events``: (gathered, encoded) events to record instead of this
        object's own (timing events of the caller: one record serves both
        the ordering and the timing, and every record costs the stream a
        few microseconds)."""
        o = dict(o)
        tenc = o.pop("tenc")
        table.sample_into(q, tq, o)
        gathered, encoded = events if events is not None else (self.gathered, self.encoded[self.slot])
        gathered.record()
        self.stream.wait_event(gathered)
        table.time_encode_into(o["ts"], tq, tenc, stream=self.stream)
        encoded.record(self.stream)
        self.used[self.slot] = encoded
        self.count += 1

    def join(self):
        import torch
        if self.used[self.slot] is not None:
            torch.cuda.current_stream().wait_event(self.used[self.slot])

    def forget(self):
        """Drop the record of earlier encodings once the device has finished
        them (after a synchronisation), so that no later join waits on an
        event recorded outside a graph being captured."""
        self.used = [None] * self.depth

    def join_all(self):
        import torch
        for k in range(self.depth):
            if self.used[k] is not None:
                torch.cuda.current_stream().wait_event(self.used[k])


def streamed_leg(w, table, b0, n, out, nbr, dev, live, host_slots=8, dev_slots=4, enc=None):
    """Steps b0 .. b0+n-1 with each batch arriving from host memory: the
    batch (queries [src | dst | neg] and times, the blocked layout) sits in a
    pinned host buffer, a second stream copies it to one of `dev_slots`
    device buffers, and the compute stream waits for that copy (an event)
    before sample + insert; the copy of a device buffer waits for the step
    that last used it (another event).  live: a host thread generates each
    batch into a ring of `host_slots` pinned buffers while the steps run (a
    slot is reused once its copy has finished); else all n batches are
    generated into pinned memory before timing.  Returns the rates."""
    import collections
    import threading

    import numpy as np
    import torch

    import synth
    import gc
    Q = 3 * w.batch
    slots = host_slots if live else n
    # one pinned buffer per batch: queries [src | dst | neg] then their times
    h_buf = torch.empty((slots, 2, Q), dtype=torch.int32, pin_memory=True)
    d_buf = torch.empty((dev_slots, 2, Q), dtype=torch.int32, device=dev)
    sizes = [w.batch_range(b0 + k)[1] - w.batch_range(b0 + k)[0] for k in range(n)]
    gen_s = [0.0]

    def fill(slot, k):
        lo, hi = w.batch_range(b0 + k)
        m = hi - lo
        hn, ht = h_buf[slot, 0].numpy(), h_buf[slot, 1].numpy().view(np.uint32)
        t0 = time.perf_counter()
        synth.host_links(w, lo, hi, out=(hn[:m], hn[m:2 * m], ht[:m], hn[2 * m:3 * m]))
        ht[m:2 * m] = ht[:m]
        ht[2 * m:3 * m] = ht[:m]
        gen_s[0] += time.perf_counter() - t0

    ready = [threading.Event() for _ in range(n)]
    free = threading.Semaphore(slots)
    if not live:
        for k in range(n):
            fill(k, k)
            ready[k].set()

    def producer():
        for k in range(n):
            free.acquire()
            fill(k % slots, k)
            ready[k].set()

    copy_stream = torch.cuda.Stream(device=dev)
    compute = torch.cuda.current_stream(dev)
    ev_copied = [torch.cuda.Event() for _ in range(n)]
    ev_free = [torch.cuda.Event() for _ in range(dev_slots)]
    pending = collections.deque()
    torch.cuda.synchronize(dev)
    th = threading.Thread(target=producer, daemon=True) if live else None
    gc.disable()
    t0 = time.perf_counter()
    if th is not None:
        th.start()
    for k in range(n):
        ready[k].wait()
        r, h, m = k % dev_slots, k % slots, sizes[k]
        with torch.cuda.stream(copy_stream):
            if k >= dev_slots:
                copy_stream.wait_event(ev_free[r])
            d_buf[r].copy_(h_buf[h], non_blocking=True)
            ev_copied[k].record(copy_stream)
        compute.wait_event(ev_copied[k])
        q, tq = d_buf[r, 0, :3 * m], d_buf[r, 1, :3 * m]
        o = {kk: v[:3 * m] for kk, v in out.items()}
        o["nbr"] = nbr[:3 * m]
        if enc is None:
            table.sample_into(q, tq, o)
            table.insert(q[:m], q[m:2 * m], tq[:m])
        else:
            enc.sample_into(table, q, tq, o)
            table.insert(q[:m], q[m:2 * m], tq[:m])
            enc.join_all()
        ev_free[r].record(compute)
        if live:
            pending.append(ev_copied[k])
            while pending and (len(pending) >= slots or pending[0].query()):
                pending.popleft().synchronize()
                free.release()
    torch.cuda.synchronize(dev)
    elapsed = time.perf_counter() - t0
    gc.enable()
    if th is not None:
        th.join()
    links = sum(sizes)
    return {"links_per_s": links / elapsed, "queries_per_s": 3 * links / elapsed,
            "ms_per_step": elapsed / n * 1e3, "steps": n, "batches": [b0, b0 + n - 1],
            "h2d_gb_per_s": 2 * 4 * Q * n / elapsed / 1e9,
            "host_generator_links_per_s": links / gen_s[0],
            "source": ("host generator thread writing each batch into a ring of pinned buffers "
                       "during the run" if live else "batches generated into pinned host memory "
                       "before timing")}


def cpu_rnn_baseline(w, first_batch, budget_s, max_batches=50, max_links=20000):
    """The CPU oracle's node-status update (fp64 GRU), single-threaded, on the
    batches the GPU times (from first_batch on; at most their first max_links
    links each) until the time budget is used.  Each batch's endpoints are
    renumbered onto a compact status array of its distinct nodes (the update
    reads and writes only those rows); statuses, link rows and renumbering
    are prepared outside the timed region."""
    import numpy as np

    import oracle
    import synth
    d, dt = synth.status_spec(w)
    W = synth.gru_weights(w)
    fw, fb = synth.time_params(w)
    rng = np.random.default_rng(7000 + w.key)
    links = updates = 0
    spent = 0.0
    b = first_batch
    while b < min(w.batches, first_batch + max_batches) and spent < budget_s:
        lo, hi = w.batch_range(b)
        hi = min(hi, lo + max_links)
        src, dst, t, _ = synth.host_links(w, lo, hi)
        nodes, inv = np.unique(np.concatenate([src, dst]), return_inverse=True)
        s_l, d_l = inv[:len(src)].astype(np.int32), inv[len(src):].astype(np.int32)
        if w.node_dim and d == w.node_dim and dt == w.node_dtype:
            st = synth.host_feature_rows(w, "node", nodes)
        else:
            x = rng.standard_normal((len(nodes), d)).astype(np.float32)
            st = synth._to_bf16_bits(x) if dt == "bf16" else x
        st = np.ascontiguousarray(st)
        ef = synth.host_feature_rows(w, "edge", np.arange(lo, hi)) if w.edge_dim else None
        t0 = time.perf_counter()
        oracle.gru_update(st, s_l, d_l, t, 0, fw, fb, ef, W)
        spent += time.perf_counter() - t0
        links += hi - lo
        updates += len(nodes)
        b += 1
    return {"value": links / spent, "unit": "links/s", "cores": 1, "kind": "oracle",
            "node_updates_per_s": updates / spent, "seconds": spent,
            "sample": f"batches {first_batch}..{b - 1} of the timed window, at most their first "
                      f"{max_links} links ({links} links, {updates} node updates), one thread, "
                      f"each batch's nodes on a compact status array"}


def graph_mode(args, w, table, start, W, K, step, update, nbr_all, nodes, ts, setup_s, enc=None):
    """The K timed steps captured in one HIP graph (every call enqueues
    kernels only; the insert and the status update keep their stream state on
    the device), then one replay timed with events on the replay stream and
    with the host clock."""
    import numpy as np
    import torch

    import paper_2402_01964_amd as nlb
    import synth
    graph = torch.cuda.CUDAGraph()
    qcount = []
    torch.cuda.synchronize()
    if enc is not None:
        enc.forget()
    t_cap = time.perf_counter()
    with torch.cuda.graph(graph):
        for k in range(K):
            b = start + W + k
            s_, d_, t_, n = step(b, nbr_all[k])
            table.insert(s_, d_, t_)
            update(b, s_, d_, t_)
            if enc is not None:
                enc.join()
            qcount.append(n)
        if enc is not None:
            enc.join_all()
    capture_s = time.perf_counter() - t_cap
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    graph.replay()
    e1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ev_s = e0.elapsed_time(e1) * 1e-3
    assert table.status() == nlb.NLB_OK
    links = sum(n // 3 for n in qcount)
    queries = sum(qcount)
    valid = int(sum(int((nbr_all[k, :qcount[k]] >= 0).sum()) for k in range(K)))
    res = {
        "metric": "interactions/s ingested + sampled queries/s; achieved HBM GB/s vs peak",
        "value": links / elapsed, "unit": "links/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": elapsed / K * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int64+f32",
        "data": "synthetic (seeded counter-based stream and features, generated in HBM)",
        "config": {"workload": w.name, "nodes": w.num_nodes, "links": w.links, "s": w.s,
                   "alpha": w.alpha, "batch": w.batch, "queries_per_batch": 3 * w.batch,
                   "d_time": w.d_time, "start_batch": start,
                   "timed_batches": [start + W, start + W + K - 1], "captured": "one HIP graph"},
        "queries_per_s": queries / elapsed,
        "ms_per_step_events": ev_s / K * 1e3,
        "valid_slot_fraction": valid / (queries * w.s),
        "capture_s": capture_s, "setup_s": setup_s,
        "value_note": "the K timed steps captured in one HIP graph and replayed once"
                      + (" (with the status update)" if args.rnn else ""),
        "encode_stream": enc is not None,
        "encode_depth": enc.depth if enc is not None else 0,
    }
    print(json.dumps(res), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for {args.gpus}); on several GPUs "
              "each would hold the table rows of its share of the node ids", file=sys.stderr)
        sys.exit(2)
    import numpy as np

    import synth
    w = synth.workload(args.workload)
    if args.cpu_plan:
        print(json.dumps(cpu_plan(w)), flush=True)
        return
    import torch

    import paper_2402_01964_amd as nlb
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.gather_probe_mb:
        rows = args.gather_probe_mb * (1 << 20) // 256
        src_t = torch.zeros((8 * rows, 128), dtype=torch.bfloat16, device=dev)
        idx = torch.randperm(8 * rows, device=dev)[:rows]
        dst_t = torch.empty((rows, 128), dtype=torch.bfloat16, device=dev)
        for _ in range(5):
            torch.index_select(src_t, 0, idx, out=dst_t)   # reads and writes gather_probe_mb MiB each
        torch.cuda.synchronize()
        del src_t, idx, dst_t
    if args.copy_probe_mb:
        n = args.copy_probe_mb * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        c = torch.empty_like(a)
        for _ in range(5):
            torch.neg(a, out=c)   # reads and writes copy_probe_mb MiB each
        torch.cuda.synchronize()
        del a, c
    K, W = args.steps, args.warmup
    start = args.start_batch
    if start is None:
        start = max(0, min(w.batches // 2, w.batches - K - W))
    if start + W + K > w.batches:
        K = max(1, w.batches - start - W)

    t_setup = time.perf_counter()
    nodes, ts = synth.device_links(w, dev)
    ef = synth.device_features(w, "edge", dev)
    nf = synth.device_features(w, "node", dev)
    fw, fb = synth.time_params(w)
    tw, tb = torch.from_numpy(fw).to(dev), torch.from_numpy(fb).to(dev)
    table = nlb.Table(w.num_nodes, w.s, w.alpha, w.table_seed, time_w=tw, time_b=tb,
                      edge_feat=ef, node_feat=nf)
    print(f"bench: {w.name}: inputs in HBM; inserting batches 0..{start - 1}", file=sys.stderr,
          flush=True)
    for b in range(start):
        s_, d_, t_, _, _ = synth.batch_views(w, nodes, ts, b)
        table.insert(s_, d_, t_)
        if (b + 1) % 1000 == 0:
            torch.cuda.synchronize()
            print(f"bench: inserted {b + 1} batches", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    Qmax = 3 * w.batch
    out = table.alloc_outputs(Qmax, want=("eid", "ts", "tenc", "efeat", "nfeat", "self"))
    nbr_all = torch.empty((K, Qmax, w.s), dtype=torch.int32, device=dev)
    enc_bytes = 4 * Qmax * w.s * w.d_time        # time encoding of one batch's retrieval
    # (not with a second hop: that launch's random table reads and the
    # encoding's write stream slow each other down more than they overlap)
    use_enc = args.encode_stream or (enc_bytes >= ENCODE_STREAM_MIN_BYTES and not args.hop2)
    enc = (EncodeStream(dev, args.encode_depth)
           if use_enc and not (args.aggregate or args.serial_encode) else None)
    outs = [out] + [table.alloc_outputs(Qmax, want=("eid", "ts", "tenc", "efeat", "nfeat", "self"))
                    for _ in range(1, enc.depth if enc is not None else 1)]
    agg_w = agg_z = None
    if args.aggregate:
        agg_w = {k: (torch.from_numpy(v.view(np.int16)) if v.dtype == np.uint16 else
                     torch.from_numpy(v)).to(dev) for k, v in synth.agg_weights(w).items()}
        agg_z = torch.empty((Qmax, nlb.AGG_HIDDEN), dtype=torch.float32, device=dev)
    hop2_out = None
    if args.hop2:
        hop2_out = table.alloc_outputs(Qmax * w.s, want=("nbr", "eid", "ts"))
    gru_w = status = None
    if args.rnn:
        d_r, dt_r = synth.status_spec(w)
        gru_w = {k: (torch.from_numpy(v.view(np.int16)) if v.dtype == np.uint16 else
                     torch.from_numpy(v)).to(dev) for k, v in synth.gru_weights(w).items()}
        if nf is not None:
            status = nf                     # the gathered node rows are the statuses
        else:
            status = torch.empty((w.num_nodes, d_r), dtype=torch.float32, device=dev)
            status.normal_(generator=torch.Generator(device=dev).manual_seed(7000 + w.key))
    setup_s = time.perf_counter() - t_setup

    def step(b, nbr_out, events=None):
        s_, d_, t_, q, tq = synth.batch_views(w, nodes, ts, b)
        n = q.numel()
        if agg_w is not None:
            table.aggregate(q, tq, agg_w, out=agg_z[:n], heads=args.heads)
            return s_, d_, t_, n
        o = {k: v[:n] for k, v in outs[enc.slot if enc is not None else 0].items()}
        o["nbr"] = nbr_out[:n]
        if enc is not None:
            enc.sample_into(table, q, tq, o, events)
        else:
            table.sample_into(q, tq, o)
        return s_, d_, t_, n

    def update(b, s_, d_, t_):
        if status is not None:
            table.rnn_update(s_, d_, t_, b * w.batch, gru_w, status)

    for k in range(W):
        s_, d_, t_, _ = step(start + k, nbr_all[0])
        table.insert(s_, d_, t_)
        update(start + k, s_, d_, t_)
        if enc is not None:
            enc.join()
    torch.cuda.synchronize()

    print(f"bench: warm-up done; timing {K} steps", file=sys.stderr, flush=True)
    if args.graph:
        return graph_mode(args, w, table, start, W, K, step, update, nbr_all, nodes, ts, setup_s, enc)
    # HIP events on the library's stream time each phase.  A recorded event
    # costs the stream a few microseconds, so a step records only those it
    # needs: its start (which also ends the previous step's last phase), the
    # end of its retrieval, and the end of the second hop / the insertion
    # only when a second hop / a status update follows.
    def mk():
        return torch.cuda.Event(enable_timing=True)
    e_start = [mk() for _ in range(K + 1)]
    e_sample = [mk() for _ in range(K)]
    e_hop2 = [mk() for _ in range(K)] if hop2_out is not None else None
    e_ins = [mk() for _ in range(K)] if status is not None else None
    # with the encoding on its own stream: its end, and the end of the
    # current stream's own work before it waits for the encoding
    e_enc = [mk() for _ in range(K)] if enc is not None else None
    e_main = [mk() for _ in range(K)] if enc is not None else None
    qcount = []
    import gc
    gc.disable()
    t0 = time.perf_counter()
    for k in range(K):
        b = start + W + k
        e_start[k].record()
        if enc is not None:
            # the encoder records e_sample (end of the table reads) and
            # e_enc (end of the encoding) as its ordering events
            s_, d_, t_, n = step(b, nbr_all[k], (e_sample[k], e_enc[k]))
        else:
            s_, d_, t_, n = step(b, nbr_all[k])
            e_sample[k].record()
        if hop2_out is not None:
            _, _, _, _, tq = synth.batch_views(w, nodes, ts, b)
            o2 = {kk: v[:n * w.s] for kk, v in hop2_out.items()}
            table.sample_hop2_into(nbr_all[k, :n], tq, o2)
            e_hop2[k].record()
        table.insert(s_, d_, t_)
        if status is not None:
            e_ins[k].record()
            update(b, s_, d_, t_)
        if enc is not None:
            e_main[k].record()
            enc.join()
        qcount.append(n)
    if enc is not None:
        enc.join_all()
    e_start[K].record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gc.enable()
    assert table.status() == nlb.NLB_OK

    def span(a, b_):
        return np.array([a[k].elapsed_time(b_[k]) for k in range(K)])
    step_end = e_main if e_main is not None else e_start[1:]
    ins_from = e_hop2 if e_hop2 is not None else e_sample
    ins_to = e_ins if e_ins is not None else step_end
    # the retrieval ends with its time encoding (on its own stream if split)
    sample_ms = span(e_start, e_enc if e_enc is not None else e_sample)
    hop2_ms = span(e_sample, e_hop2) if e_hop2 is not None else np.zeros(K)
    insert_ms = span(ins_from, ins_to)
    rnn_ms = span(e_ins, step_end) if e_ins is not None else np.zeros(K)
    links = sum(n // 3 for n in qcount)
    queries = sum(qcount)
    if agg_w is not None:
        # The aggregation writes no ids; its valid-slot counts come from a
        # replay of the timed batches' first-hop ids on a fresh table (not timed).
        replay = nlb.Table(w.num_nodes, w.s, w.alpha, w.table_seed)
        for b in range(start + W + K):
            s_, d_, t_, q, tq = synth.batch_views(w, nodes, ts, b)
            if b >= start + W:
                replay.sample_into(q, tq, {"nbr": nbr_all[b - start - W, :q.numel()]})
            replay.insert(s_, d_, t_)
        torch.cuda.synchronize()
        replay.close()
    valid = int(sum(int((nbr_all[k, :qcount[k]] >= 0).sum()) for k in range(K)))
    s_bytes = sum(sample_bytes(w, 0, n) for n in qcount) + valid * (w.row_bytes("edge") + w.row_bytes("node"))
    # With two output sets a batch's encoding overlaps the next batch's table
    # reads, so a retrieval has no span of its own: its rate is then taken
    # over the event-timed span of all K steps, inserts included (a lower
    # bound on the retrieval's own rate).
    pipelined = enc is not None and enc.depth > 1
    ret_s = (e_start[0].elapsed_time(e_start[K]) if pipelined else sample_ms.sum()) * 1e-3
    achieved = s_bytes / ret_s / 1e9
    full_bytes_per_query = sample_bytes(w, w.s, 1)
    traffic = measured_traffic(w)
    res = {
        "metric": "interactions/s ingested + sampled queries/s; achieved HBM GB/s vs peak",
        "value": links / elapsed,
        "unit": "links/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": elapsed / K * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64+f32",
        "data": "synthetic (seeded counter-based stream and features, generated in HBM)",
        "config": {"workload": w.name, "nodes": w.num_nodes, "links": w.links, "s": w.s,
                   "alpha": w.alpha, "batch": w.batch, "queries_per_batch": 3 * w.batch,
                   "d_time": w.d_time, "edge_row_bytes": w.row_bytes("edge"),
                   "node_row_bytes": w.row_bytes("node"), "start_batch": start,
                   "timed_batches": [start + W, start + W + K - 1]},
        "queries_per_s": queries / elapsed,
        "sample_kernel_queries_per_s": queries / (sample_ms.sum() * 1e-3),
        "insert_kernel_links_per_s": links / (insert_ms.sum() * 1e-3),
        "sample_ms_avg": float(sample_ms.mean()),
        "insert_ms_avg": float(insert_ms.mean()),
        "valid_slot_fraction": valid / (queries * w.s),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBPS, "traffic": traffic,
                     "traffic_unit": "bytes per nlb_sample call (rocprofv3 FETCH_SIZE + WRITE_SIZE "
                                     "of its launches, scaled by a copy kernel)",
                     "traffic_rate_gbps": (traffic / (ret_s / K) / 1e9 if traffic else None),
                     "time_basis": ("event-timed span of the K steps (the retrievals overlap each "
                                    "other and the inserts)" if pipelined else
                                    "summed event-timed spans of the K retrievals"),
                     "kernel": ("nlb_sample (sample_gather) + nlb_time_encode (tenc_stream, on a "
                                "second stream beside the insert)" if enc is not None else
                                "nlb_sample: sample_gather (+ tenc_stream on large launches "
                                "that write timestamps)"),
                     "bytes_per_launch": s_bytes / K,
                     "bytes_per_query_full_occupancy": full_bytes_per_query},
        "setup_s": setup_s,
        "encode_stream": enc is not None,
        "encode_depth": enc.depth if enc is not None else 0,
    }
    if agg_w is not None:
        fl = aggregate_flops(w, valid, queries, heads=args.heads)
        ab = aggregate_bytes(w, valid, queries)
        t_s = sample_ms.sum() * 1e-3
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        kname = aggregate_kernel(w, 3 * w.batch, cus, args.heads)
        agg_traffic = (measured_traffic(w, "nlb_aggregate")
                       if kname == "aggregate_packed" and args.heads == 1 else None)
        res["roofline"] = dict(binding_roofline(fl, ab, t_s), traffic=agg_traffic,
                               traffic_unit="bytes per nlb_aggregate launch (rocprofv3 FETCH_SIZE "
                                            "+ WRITE_SIZE, reads scaled by a random-gather kernel)",
                               kernel="nlb_aggregate: " + kname, flops_per_launch=fl / K,
                               bytes_per_launch=ab / K)
        res["aggregate_ms_avg"] = res.pop("sample_ms_avg")
        res["aggregate_kernel_queries_per_s"] = res.pop("sample_kernel_queries_per_s")
        res["value_note"] = "steps retrieve with nlb_aggregate (eq. (4), random weights)"
        res["dtype"] = "bf16-mfma+f32"
        res["config"]["heads"] = args.heads
    if hop2_out is not None:
        n_last = qcount[-1] * w.s
        last_valid = int((hop2_out["nbr"][:n_last] >= 0).sum())   # last step, after timing
        hb = sum(hop2_bytes(w, int((nbr_all[k, :qcount[k]] >= 0).sum()), qcount[k])
                 for k in range(K))
        hach = hb / (hop2_ms.sum() * 1e-3) / 1e9
        res["hop2"] = {"kernel": "sample_gather (second hop, ids only)",
                       "hop2_queries_per_s": queries * w.s / (hop2_ms.sum() * 1e-3),
                       "ms_avg": float(hop2_ms.mean()), "valid_slot_fraction_last_step":
                           last_valid / (n_last * w.s),
                       "roofline": {"bound": "hbm", "achieved": hach, "peak": PEAK_HBM_GBPS,
                                    "unit": "GB/s", "frac": hach / PEAK_HBM_GBPS}}
        res["value_note"] = "value includes the second-hop launches (--hop2)"
    if status is not None:
        # Winners per timed batch (distinct endpoints), counted after timing.
        winners = 0
        for k in range(K):
            s_, d_, _, _, _ = synth.batch_views(w, nodes, ts, start + W + k)
            winners += int(torch.unique(torch.cat([s_, d_])).numel())
        d_r = status.shape[1]
        fl = rnn_flops(w, d_r, winners)
        rb = rnn_bytes(w, d_r, status.element_size(), links, winners)
        t_s = rnn_ms.sum() * 1e-3
        res["rnn"] = {"kernels": "rnn_resolve(_merged) + rnn_select + rnn_gru_ws (or rnn_gru) + rnn_scatter",
                      "status": f"{d_r} x {str(status.dtype).replace('torch.', '')}",
                      "links_per_s": links / t_s, "node_updates_per_s": winners / t_s,
                      "ms_avg": float(rnn_ms.mean()), "updates_per_batch": winners / K,
                      "roofline": dict(binding_roofline(fl, rb, t_s), flops_per_launch=fl / K,
                                       bytes_per_launch=rb / K)}
        if enc is not None:
            res["rnn"]["timing_note"] = (
                "the update is timed from the end of the insert while the time encoding runs "
                "beside it on its own stream: its GRU pass waits for the encoding's workgroups to "
                "leave the CUs, so ms_avg and the roofline understate the update; --serial-encode "
                "times it alone")
        res["value_note"] = "value includes the node-status updates (--rnn)"
    if agg_w is None and hop2_out is None and status is None and args.streamed_steps > 0:
        b0 = start + W + K
        n_s = min(args.streamed_steps, (w.batches - b0) // 2)
        if n_s > 0:
            print(f"bench: host-streamed legs, {n_s} steps each", file=sys.stderr, flush=True)
            res["streamed"] = {
                "live_generator": streamed_leg(w, table, b0, n_s, out, nbr_all[0], dev, live=True, enc=enc),
                "staged_pinned": streamed_leg(w, table, b0 + n_s, n_s, out, nbr_all[0], dev, live=False,
                                              enc=enc),
                "note": "same step (nlb_sample + nlb_insert_batch) with each batch copied host to "
                        "device (pinned buffers, second stream, event-ordered) instead of resident "
                        "in HBM; not the headline value"}
            assert table.status() == nlb.NLB_OK
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(
            w, start + W, args.cpu_seconds,
            agg_weights=synth.agg_weights(w) if agg_w is not None else None, hop2=hop2_out is not None,
            heads=args.heads)
        if status is not None:
            print("bench: timing the CPU oracle's status update", file=sys.stderr, flush=True)
            res["rnn"]["cpu_baseline"] = cpu_rnn_baseline(w, start + W, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
