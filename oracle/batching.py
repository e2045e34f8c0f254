"""Oracle of inter-request batching: batch formation, padding, round-robin
scheduling on a simulated clock, row routing, and the merged run.

Test infrastructure only: nothing on the product path imports this module.

Paper, section 2.2.1 (Inter-Request Batching):
  * many requests are merged into one by concatenating their input tensors;
  * the core library keeps one batching queue per servable (or version);
  * the queues are scheduled round-robin onto one shared device;
  * the batching Session wrapper concatenates the inputs of several Run()
    calls, forwards them to the wrapped Run() once, and hands every caller
    its own part of the result.

The paper gives no formation rule, padding rule or clock; the readings taken
here are (each is a named choice in the design notes):
  * next-fit formation in arrival order: a batch closes when it is full, when
    the next request would overflow it (that request starts the next batch),
    when its timeout expires (measured from its first request's arrival), or
    at the end of the trace (count-only queues close there);
  * padded size P = the smallest allowed batch size >= the real size s, or
    s itself when no allowed sizes are given;
  * one serial simulated device that takes launch windows of up to W closed
    batches: when it is free and some queue holds a closed batch, it picks
    batches one at a time, each time the oldest closed batch of the next queue
    holding one (queue ids scanned cyclically from the one after the
    last-served queue), until it has W of them or none is left; every batch of
    the window is dispatched then; the device is busy with it for the sum
    over the window's queues of window_ns[queue] (a fixed time per launch
    chain) plus the sum over its batches of service_ns[queue][P] nanoseconds,
    and its batches complete window_tail_ns[queue] (summed over its queues)
    after that: a launch chain's fixed latency that the device overlaps with
    the next window. W = 1, window_ns = 0 and window_tail_ns = 0 is one batch
    at a time;
  * events at one timestamp: timeouts (queue id order), then arrivals
    (request id order), then the end-of-trace close, then dispatch;
  * within a batch, requests keep arrival order; request r's rows are rows
    [dst_row[r], dst_row[r] + n_r) of the batch, where dst_row is the
    exclusive prefix sum of the row counts of earlier requests in the batch;
    rows [s, P) are padding and are never returned to anyone.
"""
from __future__ import annotations

import collections
import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np


@dataclasses.dataclass
class QueueCfg:
    max_batch_size: int
    allowed: Sequence[int] = ()
    timeout_ns: Optional[int] = None   # None: close by count only
    bucket_len: int = 0                # > 0: takes sequences up to this length


def padded_size(s: int, allowed: Sequence[int]) -> int:
    """Smallest allowed batch size >= s; s itself if none are given."""
    if not allowed:
        return s
    for a in allowed:
        if a >= s:
            return a
    raise ValueError(f"batch of {s} rows exceeds the largest allowed size {allowed[-1]}")


def pick_queue(queues: Sequence[QueueCfg], members: Sequence[int], max_len: int) -> int:
    """Among a servable's queues (indices `members`), the one a request goes
    to: the only one, or for length-bucketed queues the smallest bucket that
    holds the request's longest sequence."""
    if len(members) == 1 and queues[members[0]].bucket_len == 0:
        return members[0]
    best = None
    for q in members:
        b = queues[q].bucket_len
        if b >= max_len and (best is None or b < queues[best].bucket_len):
            best = q
    if best is None:
        raise ValueError(f"no bucket holds a sequence of {max_len} tokens")
    return best


@dataclasses.dataclass
class Batch:
    queue: int
    reqs: List[int]
    s: int
    P: int
    close_ns: int
    dispatch_ns: int = -1
    done_ns: int = -1
    window: int = -1                # index of the device dispatch (launch window) that took it


@dataclasses.dataclass
class SimResult:
    batches: List[Batch]            # in dispatch order
    done_ns: np.ndarray             # per request
    queue_of: np.ndarray            # per request

    def latency_ns(self, arrival_ns: np.ndarray) -> np.ndarray:
        return self.done_ns - np.asarray(arrival_ns, np.int64)


def simulate(queues: Sequence[QueueCfg], req_queue: Sequence[int], arrival_ns: Sequence[int],
             n_rows: Sequence[int], service_ns: Sequence[Sequence[int]], window: int = 1,
             window_ns: Optional[Sequence[int]] = None,
             window_tail_ns: Optional[Sequence[int]] = None) -> SimResult:
    """Batch formation per queue plus round-robin dispatch on one simulated
    serial device that takes launch windows of up to `window` closed batches.
    service_ns[q][P] is the device time of a batch of padded size P from queue
    q, window_ns[q] (default 0) the fixed device time of queue q's launch
    chain in a window, window_tail_ns[q] (default 0) the further time until
    that chain's results are complete. Returns the batches in dispatch
    order."""
    if window < 1:
        raise ValueError("window must be >= 1")
    N = len(arrival_ns)
    arrival = [int(a) for a in arrival_ns]
    for i in range(1, N):
        if arrival[i] < arrival[i - 1]:
            raise ValueError("arrival times must be non-decreasing")
    nq = len(queues)
    for r in range(N):
        if not (1 <= n_rows[r] <= queues[req_queue[r]].max_batch_size):
            raise ValueError(f"request {r}: {n_rows[r]} rows")

    open_reqs: List[List[int]] = [[] for _ in range(nq)]
    open_s = [0] * nq
    open_t = [0] * nq
    closed: List[collections.deque] = [collections.deque() for _ in range(nq)]
    order: List[Batch] = []
    done = np.full(N, -1, dtype=np.int64)

    def close(q: int, t: int) -> None:
        s = open_s[q]
        closed[q].append(Batch(q, open_reqs[q], s, padded_size(s, queues[q].allowed), t))
        open_reqs[q] = []
        open_s[q] = 0

    wns = [0] * nq if window_ns is None else [int(x) for x in window_ns]
    tails = [0] * nq if window_tail_ns is None else [int(x) for x in window_tail_ns]
    last_served = -1
    n_windows = 0
    device_free = -(2 ** 62)
    end_t = arrival[-1] if N else 0
    flushed = N == 0
    nxt = 0  # next arrival to process

    def next_timeout():
        best = None
        for q in range(nq):
            T = queues[q].timeout_ns
            if T is not None and open_s[q] > 0:
                t = open_t[q] + T
                if best is None or t < best:
                    best = t
        return best

    while True:
        pending = any(closed[q] for q in range(nq))
        cands = []
        if nxt < N:
            cands.append(arrival[nxt])
        to = next_timeout()
        if to is not None:
            cands.append(to)
        if not flushed and nxt >= N:
            cands.append(end_t)
        if pending:
            # closed batches wait only while the device is busy
            cands.append(device_free)
        if not cands:
            break
        t = min(cands)
        # 1. timeouts due at t, in queue id order
        for q in range(nq):
            T = queues[q].timeout_ns
            if T is not None and open_s[q] > 0 and open_t[q] + T == t:
                close(q, t)
        # 2. arrivals at t, in request id order
        while nxt < N and arrival[nxt] == t:
            r = nxt
            q = req_queue[r]
            B = queues[q].max_batch_size
            n = int(n_rows[r])
            if open_s[q] > 0 and open_s[q] + n > B:
                close(q, t)
            if open_s[q] == 0:
                open_t[q] = t
            open_reqs[q].append(r)
            open_s[q] += n
            if open_s[q] == B:
                close(q, t)
            nxt += 1
        # 3. end of trace: count-only queues close their open batch
        if not flushed and nxt >= N and t == end_t:
            for q in range(nq):
                if queues[q].timeout_ns is None and open_s[q] > 0:
                    close(q, t)
            flushed = True
        # 4. dispatch windows while the device is free at t
        while device_free <= t and any(closed[q] for q in range(nq)):
            win: List[Batch] = []
            while len(win) < window and any(closed[q] for q in range(nq)):
                for k in range(1, nq + 1):
                    q = (last_served + k) % nq
                    if closed[q]:
                        break
                win.append(closed[q].popleft())
                last_served = q
            qs_in = sorted({b.queue for b in win})
            busy = sum(wns[q] for q in qs_in) + sum(int(service_ns[b.queue][b.P]) for b in win)
            tail = sum(tails[q] for q in qs_in)
            for b in win:
                b.dispatch_ns = t
                b.done_ns = t + busy + tail
                b.window = n_windows
                for r in b.reqs:
                    done[r] = b.done_ns
            order.extend(win)
            n_windows += 1
            device_free = t + busy
    return SimResult(order, done, np.asarray(req_queue, np.int64))


def dst_rows(n_rows_in_batch: Sequence[int]) -> np.ndarray:
    """Row offset of each request inside its batch: exclusive prefix sum."""
    out = np.zeros(len(n_rows_in_batch), dtype=np.int64)
    acc = 0
    for i, n in enumerate(n_rows_in_batch):
        out[i] = acc
        acc += int(n)
    return out


def percentile_nearest_rank(values: Sequence[int], q: float) -> int:
    """The ceil(q * N)-th smallest value (1-based), q in (0, 1]."""
    v = np.sort(np.asarray(values))
    k = max(1, int(math.ceil(q * len(v))))
    return int(v[k - 1])


# ---------------------------------------------------------------------------
# the merged run: concatenate + pad, run once, split
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Assembled:
    dense: Optional[np.ndarray] = None      # mlp / ranking: [P, d_in]
    lens: Optional[np.ndarray] = None       # ranking: [P, n_tables]
    ids: Optional[np.ndarray] = None        # ranking: concatenated ids
    tokens: Optional[np.ndarray] = None     # seqpool: [P, T, d_in]
    seq_len: Optional[np.ndarray] = None    # seqpool: [P]


def assemble(model, payloads, P: int, pad: float = 0.0, bucket_len: int = 0) -> Assembled:
    """Concatenate the requests' input tensors along the batch axis in
    arrival order and pad the batch axis to P rows with `pad` (ranking pad
    rows have empty bags). Seqpool requests are padded along time to
    bucket_len as well."""
    if model.kind == "seqpool":
        T = bucket_len
        d = model.d_in
        toks = np.full((P, T, d), pad, dtype=np.float32)
        L = np.zeros(P, dtype=np.int64)
        row = 0
        for p in payloads:
            t0 = 0
            for Ls in p.lens:
                toks[row, :Ls] = p.dense.reshape(-1, d)[t0:t0 + Ls]
                L[row] = Ls
                t0 += Ls
                row += 1
        return Assembled(tokens=toks, seq_len=L)
    d = model.d_in
    dense = np.full((P, d), pad, dtype=np.float32)
    rows = np.concatenate([p.dense.reshape(-1, d) for p in payloads])
    dense[:rows.shape[0]] = rows
    if model.kind == "mlp":
        return Assembled(dense=dense)
    lens = np.zeros((P, model.n_tables), dtype=np.int64)
    lens[:rows.shape[0]] = np.concatenate([p.lens.reshape(-1, model.n_tables) for p in payloads])
    ids = np.concatenate([p.ids for p in payloads])
    return Assembled(dense=dense, lens=lens, ids=ids)


def run_batch(omodel, payloads, P: int, pad: float = 0.0, bucket_len: int = 0) -> List[np.ndarray]:
    """Paper's batching wrapper on one batch: merge, run once, split. Returns
    each request's output rows in request order."""
    n = [int(p.lens.shape[0]) if omodel.kind == "seqpool" else int(p.dense.reshape(-1, omodel.model.d_in).shape[0])
         for p in payloads]
    Y = omodel.forward_batch(assemble(omodel.model, payloads, P, pad, bucket_len))
    off = dst_rows(n)
    return [Y[o:o + k] for o, k in zip(off, n)]
