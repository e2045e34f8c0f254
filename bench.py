#!/usr/bin/env python
"""Throughput and latency of batched inference on one MI355X.

Default workload: the ranking model - 26 sum-pooled embedding bags (ids
Zipf(1.1) over 100k-row x 64 bf16 tables, 1..20 ids per bag) plus 13 dense
features into an MLP 1677->1024->512->256->1 (ReLU, sigmoid out), bf16
weights with fp32 accumulation; 100k requests of 1..64 examples, batches of
at most 512 rows padded to {64,128,256,512}, formed by count in arrival order.
`--workload` selects one of the other synthetic workloads instead.

One step replays the whole request trace through the library: batch
formation, padded-size choice, round-robin dispatch on the simulated clock,
and every batch's device work (route -> assemble or embedding-bag -> dense
layers -> head / pooling / split), with the request payloads already resident
in HBM and the outputs left there.

Printed: one JSON line with
  * examples/s of the replay, launch windows of 64 dispatched batches;
  * p50/p99 request latency on the simulated clock, with the device modelled
    as the library runs it (launch windows whose chain, per-batch and tail
    times are measured on this GPU from lone launch chains and back-to-back
    windows; Poisson arrivals at 90% of the simulated device's capacity for
    count-only workloads, the trace's own arrivals otherwise), and a check of
    the simulated busy time against the GPU running the clock's windows;
  * the dominant kernel against its roofline (HIP events on the library's
    stream during a profiled replay; algorithmic bytes count each layer's
    weights once per launch group) with the HBM traffic from the committed
    counter passes, every kernel's figures, and for ranking the embedding
    bag against the L2 read peak and, with distinct table rows, against HBM;
  * the CPU oracle timed on one thread on a bounded sample of the same trace;
  * the serving API's rate with host payloads (PCIe in and out), never the
    headline value.
"""
import argparse
import collections
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "examples/sec per MI355X (batched MLP/embedding model); p50/p99 request latency"
HBM_PEAK_GBS = 8000.0
# L2 read peak: 8 XCDs x 16 channels x 128 bytes per clock at 2.4 GHz
L2_PEAK_GBS = 8 * 16 * 128 * 2.4
BF16_PEAK_TFLOPS = 2500.0
F32_PEAK_TFLOPS = 157.3
KERNELS = ("route", "assemble", "embbag", "gemm_bf16", "gemm_f32", "gemm_head", "mlp_tail", "head", "seqpool", "split")

DESCRIPTION = {
    "ranking": "ranking: 26 Zipf(1.1) embedding bags over 100k x 64 bf16 tables + 13 dense -> MLP "
               "1677-1024-512-256-1 (ReLU, sigmoid), bf16 weights, fp32 accumulation; 100k requests of 1-64 "
               "examples; max batch 512, allowed {64,128,256,512}",
    "small_mlp": "small MLP: fp32 64-128(ReLU)-16; 256 requests of 1-8 rows; max batch 32, allowed {8,16,32}",
    "large_mlp": "large MLP: bf16 4096-8192-8192-4096 (ReLU hidden), fp32 accumulation; 20k requests of 1-32 rows; "
                 "max batch 1024, allowed {128,256,512,1024}",
    "multi_tenant": "multi-tenant: 4 fp32 MLPs 256-1024-1024-32 + 4 ranking models on one GPU; 50k requests, "
                    "Poisson 50k/s, servable Zipf(1.0); max batch 256, no padding, 2 ms timeout",
    "ragged_seq": "ragged sequences: fp32 per-token 256-512(ReLU)-256, masked mean-pool, 256-2 softmax; 50k requests "
                  "of 1-4 sequences of 1-512 tokens; length buckets {64,128,256,512}, max 64 sequences per batch",
}
PACK_NOTE = "; token-wise layers on the real tokens packed into consecutive rows (sub-graph batching)"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def nearest_rank(v, q):
    v = np.sort(np.asarray(v))
    return int(v[max(1, int(math.ceil(q * len(v)))) - 1])


def fused_tail(m):
    """With the fused tail on, the library runs a bf16 model's last two hidden
    layers and its narrow head as one kernel (mlp_tail) when they are ReLU
    layers of 512 and 256 outputs ahead of a 256-input head."""
    L = m.layers
    return (m.dtype == "bf16" and len(L) >= 4 and L[-1].fan_out == 1 and L[-3].fan_out == 512 and
            L[-3].act == "relu" and L[-2].fan_out == 256 and L[-2].act == "relu")


def fused_head(m):
    """The library runs a bf16 model's last hidden layer of 256 outputs and
    its 256-input narrow head as one kernel (gemm_head) unless the fused
    tail takes them."""
    L = m.layers
    return m.dtype == "bf16" and len(L) >= 2 and L[-1].fan_out == 1 and L[-2].fan_out == 256 and L[-1].fan_in == 256


def algorithmic_work(w, t, a, logd, qindex, window, fused=False):
    """Algorithmic bytes / flops of one replay, per kernel. Real model
    dimensions; padded rows count as rows, since the method pads them and
    computes them. Sequence groups: padding tokens are not written by the
    assembler and 64-token blocks of them are not computed by the GEMMs (the
    pooling never reads them; with --seq-pack the layers run on the real tokens
    alone), so both count real tokens only."""
    work = collections.defaultdict(lambda: {"bytes": 0, "flops": 0})
    nb = logd["n_batches"]
    beg = logd["b_req_begin"][:nb + 1]
    reqs = logd["b_reqs"][:beg[-1]].astype(np.int64)

    def per_batch(v):  # per-request values summed over each batch
        return np.add.reduceat(v[reqs], beg[:-1]) if nb else np.zeros(0)

    n_req = np.diff(beg)
    seen_in_window = set()
    n_dense = per_batch(np.diff(a.dense_off))
    n_ids = per_batch(np.diff(a.ids_off))
    row_desc = 32
    for b in range(nb):
        q = w.queues[qindex[int(logd["b_queue"][b])]]
        m = w.models[q.servable]
        P, s = int(logd["b_padded"][b]), int(logd["b_real"][b])
        T = q.bucket_len or 1
        M = P * T
        bf16 = m.dtype == "bf16"
        lens_bytes = s * m.n_tables * 4 if m.kind == "ranking" else (s * 4 if m.kind == "seqpool" else 0)
        work["route"]["bytes"] += int(n_req[b]) * 56 + 24 + lens_bytes + P * row_desc
        if m.kind == "ranking":
            d = m.n_tables * m.emb_dim + m.n_dense
            work["embbag"]["bytes"] += (P * row_desc + s * (m.n_tables * 4 + m.n_dense * 4)
                                        + int(n_ids[b]) * (4 + m.emb_dim * 2) + P * d * 2)
        else:
            # real inputs read once; every padded row written (for sequences
            # in 64-token buckets, the real tokens only)
            Mw = int(n_dense[b]) // m.d_in if (m.kind == "seqpool" and T % 64 == 0) else M
            work["assemble"]["bytes"] += (int(n_dense[b]) * 4 + Mw * m.d_in * (2 if bf16 else 4)
                                          + (P if m.kind == "seqpool" else M) * row_desc)
        layers = m.layers[:-1] if (m.kind == "ranking" and bf16 and m.layers[-1].fan_out == 1) else m.layers
        tail = fused and fused_tail(m)
        ghead = not tail and m.kind != "seqpool" and fused_head(m)
        if tail:
            layers = m.layers[:-3]
        elif ghead:
            layers = m.layers[:-2]
        key = "gemm_bf16" if bf16 else "gemm_f32"
        Mg = int(n_dense[b]) // m.d_in if m.kind == "seqpool" else M  # rows the layers must compute
        # a launch group (one queue's batches in one launch window) reads each
        # layer's weights once, however many batches it holds
        qid = int(logd["b_queue"][b])
        first_in_group = qid not in seen_in_window
        seen_in_window.add(qid)
        if (b + 1) % window == 0:
            seen_in_window = set()
        # a chain that ends in the split writes its last layer's real rows
        # (fp32, d_out columns) straight into the requests' outputs through
        # the row map
        rows_out = m.kind != "seqpool" and len(layers) == len(m.layers)
        es = 2 if bf16 else 4
        for li, L in enumerate(layers):
            work[key]["flops"] += 2 * Mg * L.fan_in * L.fan_out
            w_bytes = L.fan_in * L.fan_out * es if first_in_group else 0
            if rows_out and li == len(layers) - 1:
                work[key]["bytes"] += Mg * L.fan_in * es + w_bytes + s * m.d_out * 4 + P * row_desc
            else:
                work[key]["bytes"] += (Mg * L.fan_in + Mg * L.fan_out) * es + w_bytes
        if tail:
            # hidden input, the two layers' and the head's weights once per
            # launch group, one output per real row, the row map
            l2, l3, hd = m.layers[-3], m.layers[-2], m.layers[-1]
            work["mlp_tail"]["flops"] += 2 * P * (l2.fan_in * l2.fan_out + l3.fan_in * l3.fan_out + hd.fan_in)
            wts = (l2.fan_in * l2.fan_out + l3.fan_in * l3.fan_out + hd.fan_in) * 2 if first_in_group else 0
            work["mlp_tail"]["bytes"] += P * l2.fan_in * 2 + wts + s * 4 + P * row_desc
        elif ghead:
            # the layer's input and weights (once per launch group), the head's
            # weights, one output per real row, the row map
            l3, hd = m.layers[-2], m.layers[-1]
            work["gemm_head"]["flops"] += 2 * Mg * l3.fan_in * l3.fan_out + 2 * P * hd.fan_in
            wts = (l3.fan_in * l3.fan_out + hd.fan_in) * 2 if first_in_group else 0
            work["gemm_head"]["bytes"] += Mg * l3.fan_in * 2 + wts + s * 4 + P * row_desc
        elif m.kind == "ranking" and len(layers) < len(m.layers):
            last = m.layers[-1]
            work["head"]["bytes"] += P * row_desc + P * last.fan_in * 2 + last.fan_in * 2 + s * 4
            work["head"]["flops"] += 2 * P * last.fan_in
        elif m.kind == "seqpool":
            D = m.head.fan_in
            work["seqpool"]["bytes"] += (int(n_dense[b]) // m.d_in) * D * 4 + P * row_desc + s * m.d_out * 4
            work["seqpool"]["flops"] += (int(n_dense[b]) // m.d_in) * D + 2 * s * D * m.d_out
    return work


def embbag_figures(w, a, logd, window, e, sample_windows=4):
    """Two bounds for the embedding-bag launches that hold where the plain
    HBM one does not (table rows hit L2 and the Infinity Cache):
      gathered bytes per launch (every id's 128-byte table row, as the
      kernel reads them) against the L2 read peak, and
      the launch's bytes with each distinct table row counted once per launch
      window (a lower bound on what must come from HBM) against the HBM peak.
    Distinct rows per window are counted on the host over the first
    `sample_windows` windows and scaled by their share of the ids."""
    m = next(m for m in w.models if m.kind == "ranking")
    nt, dim = m.n_tables, m.emb_dim
    nb = logd["n_batches"]
    beg = logd["b_req_begin"][:nb + 1]
    reqs = logd["b_reqs"][:beg[-1]]
    launches = e["launches"]
    ids_total = int(a.ids_off[-1])
    gathered = ids_total * dim * 2 / launches
    uniq = ids_s = 0
    for wi in range(min(sample_windows, -(-nb // window))):
        rs = reqs[beg[wi * window]:beg[min((wi + 1) * window, nb)]]
        lens = np.concatenate([a.lens[a.lens_off[r]:a.lens_off[r + 1]] for r in rs]).astype(np.int64)
        ids = np.concatenate([a.ids[a.ids_off[r]:a.ids_off[r + 1]] for r in rs]).astype(np.int64)
        table = np.repeat(np.tile(np.arange(nt), lens.size // nt), lens)
        uniq += np.unique(table << 32 | ids).size
        ids_s += ids.size
    per_launch = e["bytes_per_launch"]
    unique_bytes = per_launch - gathered + (uniq / ids_s) * (ids_total / launches) * dim * 2
    secs = e["avg_us"] * 1e-6
    return {"gathered_bytes_per_launch": round(gathered), "l2_read_peak_gbs": L2_PEAK_GBS,
            "gathered_gbs": round(gathered / secs / 1e9, 1), "l2_frac": round(gathered / secs / 1e9 / L2_PEAK_GBS, 4),
            "distinct_rows_per_id": round(uniq / ids_s, 4),
            "bytes_with_distinct_rows_once_per_launch": round(unique_bytes),
            "distinct_gbs": round(unique_bytes / secs / 1e9, 1),
            "hbm_frac_distinct": round(unique_bytes / secs / 1e9 / HBM_PEAK_GBS, 4),
            "sample": f"distinct (table, id) pairs of the first {min(sample_windows, -(-nb // window))} launch windows"}


def recorded_traffic(workload, kernel):
    """HBM bytes per launch from the committed counter passes, if they were
    taken on this workload with the current kernel source (else None)."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != rec.get("sha256"):
        return None
    return rec.get("workloads", {}).get(workload, {}).get(kernel)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, t, a, seconds):
    """The oracle, as it stands, on the first requests of the trace for about
    `seconds` of CPU time (model setup excluded). The per-request forward is
    too small to profit from BLAS threads (one thread measures as fast as
    many), so it runs on one thread and reports one core; the same requests
    are then run again with the BLAS threads numpy uses by default (a bounded
    second pass, at most a quarter of the time), reported beside it."""
    from oracle.models import OracleModel
    import synth
    from threadpoolctl import threadpool_info, threadpool_limits
    blas_threads = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    oms = {}

    def run(limit_s, max_n):
        n = ex = 0
        el = 0.0
        while el < limit_s and n < max_n:
            s = int(t.servable[n])
            if s not in oms:
                oms[s] = OracleModel(w.models[s], synth.model_params(w, s))
            t0 = time.perf_counter()
            oms[s].forward(a.payload(n))
            el += time.perf_counter() - t0
            ex += int(t.n_rows[n])
            n += 1
        return n, ex, el

    with threadpool_limits(limits=1):
        n, ex, el = run(seconds, t.n)
    n2, ex2, el2 = run(seconds / 4, n)
    return {"value": ex / el, "unit": "examples/s", "cores": 1, "kind": "oracle", "requests": n,
            "sample": f"first {n} requests ({ex} examples) of the same trace, unbatched fp64 forward per request "
                      f"on one thread, {el:.1f} s",
            "cpu_model": cpu_model(),
            "blas_threads": {"value": ex2 / el2, "cores": int(blas_threads),
                             "sample": f"first {n2} requests ({ex2} examples), {el2:.1f} s"}}


def gpu_prefix_rate(dep, dt, n, reps=5):
    """The GPU's examples/s over the first n requests of the trace (the CPU
    oracle's sample), replayed in the bench's launch configuration with the
    payloads in HBM: wall time of `reps` replays, synchronized on both sides."""
    import torch
    k = min(n, dt.n)

    def cut(x, m):
        return None if x is None else x[:m]
    go = dep.sched.prepare_sim_run(
        dep.servables, dt.servable[:k], dt.arrival_ns[:k], dt.n_rows[:k], cut(dt.max_len, k),
        dense=dt.dense, dense_off=dt.dense_off[:k + 1], lens=dt.lens, lens_off=cut(dt.lens_off, k + 1),
        ids=dt.ids, ids_off=cut(dt.ids_off, k + 1), out=dt.out, out_off=dt.out_off[:k + 1])
    go()
    dep.sched.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        go()
    dep.sched.sync()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return {"value": round(int(dt.n_rows[:k].sum()) * reps / wall, 1), "unit": "examples/s", "requests": k,
            "sample": f"first {k} requests, replayed {reps} times in the bench's launch configuration"}


def cpu_latency(w, t, ns_per_example, n_max=20_000):
    """Per-request latency if the CPU oracle served the trace: one server,
    requests run unbatched in arrival order (FIFO), each taking n_r times the
    oracle's measured time per example. Count-only workloads: Poisson arrivals
    at rho x this server's capacity (rho 0.5 and 0.9), as for the GPU; workloads
    with batch timeouts: the trace's own arrivals, where a utilization above 1
    means the queue grows without bound over the trace (reported as unstable,
    with the percentiles over the simulated requests)."""
    import synth
    n = min(n_max, t.n)
    svc = t.n_rows[:n].astype(np.float64) * ns_per_example

    def fifo(arrival):
        arrival = np.asarray(arrival[:n], np.float64)
        lat = np.empty(n)
        free = -np.inf
        for r in range(n):
            free = max(arrival[r], free) + svc[r]
            lat[r] = free - arrival[r]
        return round(nearest_rank(lat, 0.5) / 1e3, 1), round(nearest_rank(lat, 0.99) / 1e3, 1)
    cap = 1e9 / float(svc.mean())
    out = {"model": "one CPU server, requests unbatched in arrival order, n_r x the measured time per example",
           "requests": n, "ns_per_example": round(ns_per_example, 1), "capacity_req_s": round(cap, 1)}
    if any(q.timeout_ns is not None for q in w.queues):
        util = w.rate_per_s / cap
        p50, p99 = fifo(t.arrival_ns)
        out["trace_arrivals"] = {"arrival_rate_req_s": w.rate_per_s, "utilization": round(util, 2),
                                 "unstable": bool(util >= 1.0), "p50_us": p50, "p99_us": p99}
    else:
        for rho in (0.5, 0.9):
            p50, p99 = fifo(synth.trace(w, n, rate_per_s=rho * cap).arrival_ns)
            out[f"rho{rho}"] = {"arrival_rate_req_s": round(rho * cap, 1), "utilization": rho,
                                "p50_us": p50, "p99_us": p99}
    return out


def serving_rate(w, t, a, ctx, models, n, seq_pack=False, window=1, tables=None, alpha=None, tail=None, rate=None):
    """The serving API with host payloads: the first n requests submitted in
    arrival order from host memory (rb_submit copies them), every launch
    window run as soon as the simulated clock dispatches it (rb_run_window:
    the window's payloads staged to HBM in one copy, one launch chain per
    queue, outputs copied back over PCIe), the rest flushed, and every
    request's rows collected on the host (rb_collect). With the calibrated
    service tables and arrivals at `rate` (above the device's capacity) the
    clock keeps a backlog, so windows fill up to `window` batches. Wall time
    from the first submit to the last collect, Python call overhead
    included; timed on a second pass over the same requests, after a first
    one has sized the scheduler's staging buffers."""
    import torch
    import synth
    from paper_1712_06139_amd import rb
    from paper_1712_06139_amd.deploy import Deployment
    n = min(n, t.n)
    arrival = t.arrival_ns if rate is None else synth.trace(w, rate_per_s=rate).arrival_ns
    dep = Deployment(w, ctx, device=True, models=models, seq_pack=seq_pack, window_batches=window,
                     service_ns=tables, window_ns=alpha, window_tail_ns=tail)
    sizes = []
    try:
        payloads = [a.payload(r) for r in range(n)]
        qs = [dep.queue_for(t, r) for r in range(n)]
        d_out = [dep.models[int(t.servable[r])].d_out for r in range(n)]
        sched = dep.sched

        def drain():
            while True:
                win = sched.run_window()
                if win is None:
                    return
                sizes.append(len(win))

        def one_pass(t_off):
            # the same requests again, later on the same clock
            ids = []
            for r in range(n):
                p = payloads[r]
                ids.append(sched.submit(qs[r], int(t.n_rows[r]), p.dense, p.lens, p.ids,
                                        arrival_ns=t_off + int(arrival[r])))
                if r + 1 == n or arrival[r + 1] != arrival[r]:
                    drain()
            for q, qc in zip(dep.queues, w.queues):
                if qc.timeout_ns is None:
                    rb.check(rb.lib().rb_flush(q.h), "rb_flush")
            end = t_off + int(arrival[n - 1]) + 10 ** 15
            sched.advance(end)
            drain()
            sched.sync()
            rows = 0
            for r in range(n):
                rows += sched.collect(ids[r], int(t.n_rows[r]), d_out[r]).shape[0]
            return rows, end

        # a first pass sizes the scheduler's staging buffers; the second is timed
        _, end = one_pass(0)
        sizes.clear()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rows, _ = one_pass(end + 1)
        el = time.perf_counter() - t0
    finally:
        dep.destroy()
    ex = int(t.n_rows[:n].sum())
    assert rows == ex
    return {"value": round(ex / el, 1), "unit": "examples/s", "requests": n, "examples": ex,
            "seconds": round(el, 3), "window_batches": window, "windows": len(sizes),
            "mean_batches_per_window": round(float(np.mean(sizes)), 2) if sizes else 0.0,
            "arrival_rate_req_s": None if rate is None else round(rate, 1),
            "path": "host payloads: rb_submit -> rb_run_window (the clock's launch windows: one staged copy, "
                    "one launch chain per queue, PCIe in and out) -> rb_collect"}


def _subset(t, a, idx):
    """Requests idx (ascending) of trace t as a trace and arenas of their own
    (slices copied so that each request's slice stays contiguous)."""
    import synth

    def cat(arr, off):
        parts = [arr[off[r]:off[r + 1]] for r in idx]
        o = np.zeros(len(idx) + 1, dtype=np.int64)
        np.cumsum([len(x) for x in parts], out=o[1:])
        return (np.concatenate(parts) if parts else arr[:0]), o

    dense, doff = cat(a.dense, a.dense_off)
    lens, loff = cat(a.lens, a.lens_off)
    ids, ioff = cat(a.ids, a.ids_off)
    seq_lens = seq_off = None
    if t.seq_lens is not None:
        seq_lens, seq_off = cat(t.seq_lens, t.seq_off)
    st = synth.Trace(t.workload, np.zeros(len(idx), dtype=t.servable.dtype), t.arrival_ns[idx], t.n_rows[idx],
                     seq_lens, seq_off)
    return st, synth.Arenas(dense, lens, ids, doff, loff, ioff)


def version_swap(w, t, a, dt, ctx, args):
    """Version transitions under load (availability-preserving policy): a
    loader thread keeps building new versions of the largest servable while
    the main thread replays the trace; after each step a loaded version
    replaces the old one (rb_queue_set_model) and the old one is destroyed
    (freed on the library's deleter thread). Step times with loading against
    the same deployment's steps without it."""
    import threading
    import synth
    from paper_1712_06139_amd.deploy import Deployment

    def size(s):
        p = synth.model_params(w, s)
        return sum(W.size for W, _ in p.weights) + sum(T.size for T in p.tables)
    S = max(range(len(w.models)), key=size)
    versions = [synth.model_params(w, S), synth.next_version(synth.model_params(w, S))]
    dep = Deployment(w, ctx, device=True, window_batches=args.window, n_streams=args.streams, seq_pack=args.seq_pack)
    st = {"ready": None, "stop": False, "load_s": []}

    def step():
        t0 = time.perf_counter()
        dep.replay(dt)
        dep.sched.sync()
        return (time.perf_counter() - t0) * 1e3

    def loader():
        v = 1
        while not st["stop"]:
            if st["ready"] is None:
                t0 = time.perf_counter()
                m = dep.build_model(S, versions[v % 2])
                st["load_s"].append(time.perf_counter() - t0)
                st["ready"] = m
                v += 1
            else:
                time.sleep(0.001)

    try:
        for _ in range(2):
            step()
        idle = [step() for _ in range(args.version_swap)]
        th = threading.Thread(target=loader)
        th.start()
        busy, swaps, t_end = [], 0, time.perf_counter() + 60
        while (len(busy) < args.version_swap or swaps < 3) and time.perf_counter() < t_end:
            busy.append(step())
            m = st["ready"]
            if m is not None:
                dep.swap(S, m).destroy()
                st["ready"] = None
                swaps += 1
        st["stop"] = True
        th.join()
        if st["ready"] is not None:
            st["ready"].destroy()
    finally:
        dep.destroy()

    def pct(v, q):
        return round(float(np.percentile(v, q)), 3)
    return {"policy": "availability-preserving", "servable": S, "versions_swapped": swaps,
            "load_ms_mean": round(1e3 * float(np.mean(st["load_s"])), 1) if st["load_s"] else None,
            "steps_idle": len(idle), "steps_loading": len(busy),
            "ms_per_step_idle": {"p50": pct(idle, 50), "p99": pct(idle, 99), "max": round(max(idle), 3)},
            "ms_per_step_loading": {"p50": pct(busy, 50), "p99": pct(busy, 99), "max": round(max(busy), 3)}}


def chain_model_fit(c1, T1, TW, nb, nw):
    """The launch-window device model from three timings: c1 a lone batch's
    chain (b + S + c), T1 one batch per window back to back (b + S per
    batch), TW nb batches in nw windows back to back (nw b + nb S). Returns
    (S, b, c): the per-batch time, the chain's fixed device time and its
    tail, clamped at S >= 1 ns and b, c >= 0."""
    S = max(1.0, (TW - nw * T1) / (nb - nw)) if nb > nw else T1
    return S, max(0.0, T1 - S), max(0.0, c1 - T1)


def _chain_ns(sched, run, reps):
    """Median device time (ns) of `run` (one replay), each repetition on its
    own: the device drained before and after it, HIP events on the
    scheduler's stream around it (the library's host work of building and
    enqueueing the chain included, as a served batch would see it; the
    binding's argument marshalling done beforehand)."""
    import torch
    st = torch.cuda.ExternalStream(sched.stream())
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    v = []
    for _ in range(reps):
        sched.sync()
        torch.cuda.synchronize()
        e0.record(st)
        run()
        e1.record(st)
        sched.sync()
        torch.cuda.synchronize()
        v.append(e0.elapsed_time(e1) * 1e6)
    return int(np.median(v))


def calibrate_latency(w, t, a, dt, ctx, dep, window, seq_pack=False, n_streams=1):
    """Per-request latency on the simulated clock (nearest-rank p50 / p99),
    with the device modelled as the library runs it: launch windows of up to
    `window` closed batches; a window holds the device for a fixed chain time
    b per queue plus S(P) per batch of padded size P, and its results are
    complete a tail time c per queue after that (the chain's fixed latency,
    which the device overlaps with the next window: consecutive windows of a
    model alternate between two launch lanes). All three are measured on this
    GPU, in the bench's stream configuration, for every queue and allowed size
    P (or B/8, B/4, B/2 and B, interpolated in between, for queues that do
    not pad), from the queue's own requests run through a queue that pads
    every batch to P:
      c1     the median of 20 isolated launch chains of one batch (a lone
             batch's latency): c1 = b + S(P) + c;
      T1     up to 256 batches replayed back to back one per window: per
             batch, T1 = b + S(P);
      TW     n batches replayed back to back in m windows of `window`
             batches, as the throughput replay runs them: TW = m b + n S(P)
             (median of 3 timings).
    b and c are averaged over P. The no-device scheduler replays arrivals with
    these tables: Poisson arrivals at rho x the simulated device's capacity
    for count-only workloads, the trace's own arrivals for workloads with
    batch timeouts. Finally those arrivals are replayed on the GPU running
    exactly the clock's windows, and the measured time is compared with the
    simulated device-busy time."""
    import dataclasses
    import synth
    import torch
    from paper_1712_06139_amd import rb
    from paper_1712_06139_amd.deploy import Deployment
    qsel = np.array([dep.qindex[dep.queue_for(t, r).id] for r in range(t.n)])
    tables, alphas, tails, measured = [], [], [], {}
    for qi, q in enumerate(w.queues):
        m_idx = q.servable
        mine = np.nonzero(qsel == qi)[0]
        sizes = sorted(set(q.allowed)) if q.allowed else sorted(
            {max(q.max_batch_size // 8, 1), q.max_batch_size // 4, q.max_batch_size // 2, q.max_batch_size})
        sizes = [P for P in sizes if P >= int(t.n_rows[mine].max(initial=1))]
        if len(w.queues) == 1:
            idx = mine[:20_000]  # a prefix of the trace, already in device memory
        else:
            # a copied subset: up to 3000 requests and about 256 MB of payload
            cum = np.cumsum(np.diff(a.dense_off)[mine])
            idx = mine[:max(1, min(3000, int(np.searchsorted(cum, 64 << 20))))]
        prefix = bool(len(idx)) and idx[-1] == len(idx) - 1
        if prefix:
            st = synth.trace(w, len(idx))
            sa = None
        else:
            st, sa = _subset(t, a, idx)
        fit = {}
        for P in sizes:
            # requests per batch when batches close at P rows (next-fit)
            ends, acc = [], 0
            for r_, nr in enumerate(st.n_rows[:len(idx)]):
                if acc + int(nr) > P:
                    ends.append(r_)
                    acc = 0
                acc += int(nr)
            ends.append(len(idx))
            nb = len(ends)
            nw = -(-nb // window)
            reps = max(1, -(-8 // nw))  # at least 8 windows back to back
            n1 = min(nb, 256)
            cw = synth.Workload(w.name, w.wid, (w.models[m_idx],),
                                (synth.Queue(0, P, (P,), None, q.bucket_len),), len(idx), w.rows, w.rate_per_s)
            times = {}
            for win in (1, window):
                cdep = Deployment(cw, ctx, device=True, window_batches=win, models=[dep.models[m_idx]],
                                  seq_pack=seq_pack, n_streams=n_streams)
                try:
                    if prefix:
                        out_off = cdep.out_offsets(st)
                        out = torch.empty(int(out_off[-1]), dtype=torch.float32, device="cuda")

                        def prep(k, cdep=cdep, out=out, out_off=out_off):
                            return cdep.sched.prepare_sim_run(
                                cdep.servables, np.zeros(k, np.int32), np.zeros(k, np.int64), st.n_rows[:k],
                                None if st.seq_lens is None else cdep.max_len(st)[:k], dense=dt.dense,
                                dense_off=a.dense_off[:k + 1], lens=dt.lens,
                                lens_off=None if a.lens.size == 0 else a.lens_off[:k + 1], ids=dt.ids,
                                ids_off=None if a.ids.size == 0 else a.ids_off[:k + 1], out=out,
                                out_off=out_off[:k + 1])
                    else:
                        sdt = cdep.upload(st, sa)

                        def prep(k, cdep=cdep, sdt=sdt):
                            return cdep.sched.prepare_sim_run(
                                cdep.servables, np.zeros(k, np.int32), np.zeros(k, np.int64), sdt.n_rows[:k],
                                None if sdt.max_len is None else sdt.max_len[:k], dense=sdt.dense,
                                dense_off=sdt.dense_off[:k + 1], lens=sdt.lens,
                                lens_off=None if sdt.lens_off is None else sdt.lens_off[:k + 1], ids=sdt.ids,
                                ids_off=None if sdt.ids_off is None else sdt.ids_off[:k + 1], out=sdt.out,
                                out_off=sdt.out_off[:k + 1])
                    # the calls' arguments are marshalled beforehand, so the
                    # timings hold the library call and the device work only
                    if win == 1:
                        k1 = ends[n1 - 1]
                        run1, runk = prep(ends[0]), prep(k1)
                        runk()
                        times["c1"] = _chain_ns(cdep.sched, run1, 20)
                        times["T1"] = _chain_ns(cdep.sched, runk, 3) / n1
                    else:
                        runa = prep(len(idx))
                        runa()
                        times["TW"] = _chain_ns(cdep.sched, lambda: [runa() for _ in range(reps)], 3) / reps
                finally:
                    cdep.destroy()
            S, b_, c_ = chain_model_fit(times["c1"], times["T1"], times["TW"], nb, nw)
            fit[P] = {"S": S, "b": b_, "c": c_, "c1": times["c1"], "T1": times["T1"], "TW": times["TW"],
                      "batches": nb, "windows": nw}
        ps = sorted(fit)
        alpha = int(np.mean([fit[P]["b"] for P in ps]))
        tail = int(np.mean([fit[P]["c"] for P in ps]))
        svc = np.zeros(q.max_batch_size + 1, dtype=np.int64)
        for s_ in range(1, q.max_batch_size + 1):
            if q.allowed:
                svc[s_] = int(fit[min(P for P in ps if P >= s_)]["S"])
            else:
                svc[s_] = int(np.interp(s_, ps, [fit[P]["S"] for P in ps]))
        svc[0] = svc[1]
        tables.append(svc.tolist())
        alphas.append(alpha)
        tails.append(tail)
        us = lambda v: round(v / 1e3, 2)
        measured[f"queue{qi}"] = {"chain_us": us(alpha), "tail_us": us(tail),
                                  "per_batch_us": {str(P): us(fit[P]["S"]) for P in ps},
                                  "lone_batch_chain_us": {str(P): us(fit[P]["c1"]) for P in ps},
                                  "back_to_back_one_per_window_us": {str(P): us(fit[P]["T1"]) for P in ps},
                                  "back_to_back_window_us": {str(P): us(fit[P]["TW"] / fit[P]["windows"])
                                                             for P in ps}}
    lctx = rb.Ctx(-1)
    ld = Deployment(w, lctx, device=False, service_ns=tables, window_ns=alphas, window_tail_ns=tails,
                    window_batches=window, with_params=False)
    lat = {"clock": "simulated", "device_model": f"launch windows of up to {window} batches: chain time per queue "
                                                  "+ time per batch of device occupancy, and a chain tail until the "
                                                  "results are complete; fitted to a lone batch's launch chain and to "
                                                  "back-to-back windows of one and of the full window of batches",
           "service": measured}

    def busy_of(lg):
        # simulated device occupancy of every launch window (the batches of a
        # window share its dispatch time): chain times of its queues plus its
        # batches' times; the tails overlap the next window
        wins = collections.defaultdict(list)
        for qid, P, d0 in zip(lg["b_queue"].tolist(), lg["b_padded"].tolist(), lg["b_dispatch_ns"].tolist()):
            wins[d0].append((ld.qindex[qid], P))
        busy = 0
        for members in wins.values():
            busy += sum(alphas[qi] for qi in {m[0] for m in members}) + sum(tables[qi][P] for qi, P in members)
        return busy, len(wins)

    def pct(lg, tr):
        v = lg["req_done_ns"] - tr.arrival_ns
        return round(nearest_rank(v, 0.5) / 1e3, 2), round(nearest_rank(v, 0.99) / 1e3, 2)
    try:
        timed = any(q.timeout_ns is not None for q in w.queues)
        min_chain = min(min(v["lone_batch_chain_us"].values()) for v in measured.values())
        lat["shortest_lone_batch_chain_us"] = min_chain
        if timed:
            check_tr = t
            lg = ld.replay_meta(t)
            busy, nw = busy_of(lg)
            span = int(lg["req_done_ns"].max() - t.arrival_ns.min())
            p50, p99 = pct(lg, t)
            lat["trace_arrivals"] = {"arrival_rate_req_s": w.rate_per_s, "utilization": round(busy / span, 3),
                                     "windows": nw, "mean_batches_per_window": round(lg["n_batches"] / nw, 2),
                                     "p50_us": p50, "p99_us": p99}
        else:
            sat = dataclasses.replace(t, arrival_ns=np.zeros(t.n, np.int64))
            busy, _ = busy_of(ld.replay_meta(sat))
            cap = t.n / (busy * 1e-9)
            lat["capacity_req_s"] = round(cap, 1)
            lat["capacity_examples_s"] = round(int(t.n_rows.sum()) / (busy * 1e-9), 1)
            for rho in (0.5, 0.9):
                tr = synth.trace(w, rate_per_s=rho * cap)
                lg = ld.replay_meta(tr)
                b_, nw = busy_of(lg)
                p50, p99 = pct(lg, tr)
                lat[f"rho{rho}"] = {"arrival_rate_req_s": round(rho * cap, 1), "utilization": rho, "windows": nw,
                                    "mean_batches_per_window": round(lg["n_batches"] / nw, 2),
                                    "p50_us": p50, "p99_us": p99}
                check_tr = tr
        # the same arrivals on the GPU, running exactly the clock's windows
        cdep = Deployment(w, ctx, device=True, window_batches=window, service_ns=tables, window_ns=alphas,
                          window_tail_ns=tails, clocked_windows=True, models=dep.models, seq_pack=seq_pack,
                          n_streams=n_streams)
        try:
            cdt = dataclasses.replace(dt, arrival_ns=check_tr.arrival_ns)
            lg = cdep.replay(cdt)
            cdep.sched.sync()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            lg = cdep.replay(cdt)
            cdep.sched.sync()
            el = time.perf_counter() - t0
            busy, nw = busy_of(lg)
            lat["model_check"] = {"arrivals": "rho0.9" if not timed else "trace", "windows": nw,
                                  "simulated_busy_ms": round(busy / 1e6, 3), "measured_ms": round(el * 1e3, 3),
                                  "measured_over_simulated": round(el * 1e9 / busy, 3)}
        finally:
            cdep.destroy()
    finally:
        ld.destroy()
        lctx.destroy()
    return lat, tables, alphas, tails


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="ranking", choices=sorted(DESCRIPTION))
    ap.add_argument("--window", type=int, default=64, help="dispatched batches per launch window")
    ap.add_argument("--version-swap", type=int, default=0,
                    help="also time this many steps while new versions of the largest servable load and swap in")
    ap.add_argument("--seq-pack", action="store_true",
                    help="sequence models: pack the real tokens of each launch group (no time padding)")
    ap.add_argument("--emb-dedup", action="store_true",
                    help="ranking models: gather each distinct table row of a 64-row block once (rb_k_embbag_dedup)")
    ap.add_argument("--fused-tail", action="store_true",
                    help="run the ranking MLP's last two layers and head as one kernel (rb_k_mlp_tail)")
    ap.add_argument("--streams", type=int, default=8,
                    help="HIP streams for concurrent launch chains of different models")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-latency", action="store_true")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache profiled replay")
    ap.add_argument("--serving-requests", type=int, default=20000,
                    help="also time the serving API with host payloads on this many requests (0: skip)")
    ap.add_argument("--sweep-windows", default="", help="comma list: also time these windows (stderr)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="first run one plain elementwise copy of this many MiB (fp32), a known-size kernel "
                         "for scaling hardware byte counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one MI355X only: batching serves independent requests, so more GPUs are "
              "independent replicas (no collectives); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_1712_06139_amd import rb
    from paper_1712_06139_amd.deploy import Deployment

    assert torch.cuda.is_available(), "needs a GPU"
    if args.copy_probe_mb:
        n = args.copy_probe_mb * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        log(f"copy probe: read {n * 4} B, wrote {n * 4} B")
        del src, dst
    w = synth.workload(args.workload)
    t = synth.trace(w)
    examples = int(t.n_rows.sum())
    log(f"{w.name}: generating {t.n} requests ({examples} rows)")
    t0 = time.time()
    a = synth.arenas(t)
    log(f"payloads drawn in {time.time() - t0:.1f} s; building models")
    ctx = rb.Ctx(0)
    shared = {}

    def make(window, profile=False, n_streams=1):
        d = Deployment(w, ctx, device=True, window_batches=window, profile=profile, models=shared.get("m"),
                       n_streams=n_streams, seq_pack=args.seq_pack, emb_dedup=args.emb_dedup,
                       fused_tail=args.fused_tail)
        shared.setdefault("m", d.models)
        return d

    dep = make(args.window, n_streams=args.streams)
    dt = dep.upload(t, a)
    log("uploaded; warmup")
    for _ in range(args.warmup):
        dep.replay(dt)
        dep.sched.sync()
    stream = torch.cuda.ExternalStream(dep.sched.stream())
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        logd = dep.replay(dt)
    ev1.record(stream)
    dep.sched.sync()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dev_ms = ev0.elapsed_time(ev1)
    ms_per_step = wall * 1e3 / args.steps
    value = examples * args.steps / wall
    n_batches = int(logd["n_batches"])
    log(f"timed {args.steps} steps: {ms_per_step:.2f} ms/step (device {dev_ms / args.steps:.2f} ms), "
        f"{value / 1e6:.2f} M rows/s, {n_batches} batches/step")

    # profiled replay: per-kernel durations from HIP events around each launch,
    # on one stream so that no other chain shares the device meanwhile
    pdep = make(args.window, profile=1)
    pdep.replay(dt)
    pdep.sched.sync()
    work = algorithmic_work(w, t, a, logd, dep.qindex, args.window, args.fused_tail)
    kernels = {}
    for k in KERNELS:
        n, ms = pdep.sched.kernel_stats(k)
        if n == 0:
            continue
        e = {"launches": n, "total_ms": round(ms, 4), "avg_us": round(ms * 1e3 / n, 3)}
        wk = work.get(k, {})
        if wk.get("bytes"):
            e["gbs"] = round(wk["bytes"] / (ms * 1e-3) / 1e9, 1)
        if wk.get("flops"):
            e["tflops"] = round(wk["flops"] / (ms * 1e-3) / 1e12, 2)
        kernels[k] = e
    pdep.destroy()
    if not args.no_cold:
        # the same replay with every launch preceded by a 512 MB read (cold L2
        # and Infinity Cache); the rates above are the warm, steady-state ones
        cdep = make(args.window, profile=2)
        cdep.replay(dt)
        cdep.sched.sync()
        for k, e in kernels.items():
            n, ms = cdep.sched.kernel_stats(k)
            if n == 0:
                continue
            e["cold_avg_us"] = round(ms * 1e3 / n, 3)
            wk = work.get(k, {})
            if wk.get("bytes"):
                e["cold_gbs"] = round(wk["bytes"] / (ms * 1e-3) / 1e9, 1)
        cdep.destroy()
    emb = None
    if "embbag" in kernels:
        ke = dict(kernels["embbag"])
        ke["bytes_per_launch"] = work["embbag"]["bytes"] / ke["launches"]
        emb = embbag_figures(w, a, logd, args.window, ke)
        log(f"embbag: {json.dumps(emb)}")
    dom = max(kernels, key=lambda k: kernels[k]["total_ms"])
    dk, wk = kernels[dom], work[dom]
    if dom.startswith("gemm") or dom == "mlp_tail":
        peak = F32_PEAK_TFLOPS if dom == "gemm_f32" else BF16_PEAK_TFLOPS
        ach = wk["flops"] / (dk["total_ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4)}
        roof["algorithmic_flops_per_launch"] = round(wk["flops"] / dk["launches"])
    elif dom == "embbag":
        # the gathered table rows are mostly L2 / Infinity Cache hits, so the
        # bytes that must cross HBM are the launch's other bytes plus each
        # distinct table row once; the gathered-bytes rate against the L2 peak
        # is in embbag_roofline
        per_launch = emb["bytes_with_distinct_rows_once_per_launch"]
        ach = per_launch / (dk["avg_us"] * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "algorithmic_bytes_per_launch": per_launch,
                "bytes_note": "distinct table rows once per launch window"}
    else:
        ach = wk["bytes"] / (dk["total_ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4)}
        roof["algorithmic_bytes_per_launch"] = round(wk["bytes"] / dk["launches"])
    roof["traffic"] = recorded_traffic(w.name + ("_packed" if args.seq_pack and w.name == "ragged_seq" else ""), dom)
    if "cold_avg_us" in dk:
        roof["cold"] = {"avg_launch_us": dk["cold_avg_us"],
                        "achieved": round(roof["achieved"] * dk["avg_us"] / dk["cold_avg_us"], 2),
                        "note": "each launch preceded by a 512 MB read (L2 and Infinity Cache evicted)"}
        roof["cold"]["frac"] = round(roof["cold"]["achieved"] / roof["peak"], 4)
    roof["traffic_unit"] = "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-probe scaled)"
    roof["kernel"] = dom
    roof["launches_per_step"] = dk["launches"]
    roof["avg_launch_us"] = dk["avg_us"]
    log(f"kernels: {json.dumps(kernels)}")

    for sw in [int(x) for x in args.sweep_windows.split(",") if x]:
        d2 = make(sw)
        d2.replay(dt)
        d2.sched.sync()
        torch.cuda.synchronize()
        s0 = time.perf_counter()
        for _ in range(2):
            d2.replay(dt)
        d2.sched.sync()
        el = (time.perf_counter() - s0) / 2
        log(f"window {sw}: {el * 1e3:.2f} ms/step, {examples / el / 1e6:.2f} M rows/s")
        d2.destroy()

    latency, tables, alphas, tails = None, None, None, None
    if not args.no_latency:
        latency, tables, alphas, tails = calibrate_latency(w, t, a, dt, ctx, dep, args.window, args.seq_pack,
                                                           args.streams)
        log(f"latency: {json.dumps(latency)}")

    serving = None
    if args.serving_requests > 0:
        log(f"serving API with host payloads ({args.serving_requests} requests)")
        # offered load above the simulated device's capacity: the clock keeps
        # a backlog, so its launch windows fill up
        cap = None if latency is None else latency.get("capacity_req_s")
        serving = serving_rate(w, t, a, ctx, shared["m"], args.serving_requests, args.seq_pack,
                               window=args.window if latency is not None else 1, tables=tables, alpha=alphas,
                               tail=tails, rate=None if cap is None else 2.0 * cap)
        log(f"serving: {json.dumps(serving)}")

    swap = None
    if args.version_swap > 0:
        log(f"version transitions under load ({args.version_swap} steps)")
        swap = version_swap(w, t, a, dt, ctx, args)
        log(f"version swap: {json.dumps(swap)}")

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle")
        cpu = cpu_baseline(w, t, a, args.cpu_seconds)
        cpu["latency"] = cpu_latency(w, t, 1e9 / cpu["value"])
        cpu["gpu_same_sample"] = gpu_prefix_rate(dep, dt, cpu["requests"])
        log(f"gpu on the cpu sample: {json.dumps(cpu['gpu_same_sample'])}")
        log(f"cpu latency: {json.dumps(cpu['latency'])}")

    dtypes = {m.dtype for m in w.models}
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "examples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dtypes.pop() if len(dtypes) == 1 else "bf16+f32", "data": "synthetic",
        "config": {"workload": DESCRIPTION[w.name] + (PACK_NOTE if args.seq_pack and w.name == "ragged_seq" else ""),
                   "requests_per_step": t.n, "examples_per_step": examples,
                   "batches_per_step": n_batches, "window_batches": args.window, "streams": args.streams,
                   "parallelism": "single GPU"},
        "latency": latency,
        "p50_us": None if latency is None else latency.get("rho0.9", latency.get("trace_arrivals"))["p50_us"],
        "p99_us": None if latency is None else latency.get("rho0.9", latency.get("trace_arrivals"))["p99_us"],
        "device_ms_per_step": round(dev_ms / args.steps, 3),
        "kernels": kernels,
        "roofline": roof,
        **({"embbag_roofline": emb} if emb is not None else {}),
        "cpu_baseline": cpu,
        "serving_pcie": serving,
        **({"version_swap": swap} if swap is not None else {}),
    }
    print(json.dumps(out), flush=True)
    dep.destroy()


if __name__ == "__main__":
    main()
