"""Pins of the oracle's batch formation and scheduling: hand-worked traces,
brute force over every order-preserving partition of tiny traces (against a
declarative statement of the closing rules), closed-form batch counts,
invariants of the dispatch log, and the sample-path form of Little's law."""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import batching as ob


def _run_case(c):
    qs = [ob.QueueCfg(q["max_batch_size"], tuple(q["allowed"]), q["timeout_ns"]) for q in c["queues"]]
    req = c["requests"]
    return ob.simulate(qs, [r[1] for r in req], [r[0] for r in req], [r[2] for r in req], c["service_ns"],
                       c.get("window", 1), c.get("window_ns"), c.get("window_tail_ns"))


def test_hand_worked_schedules(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "schedule_cases.json")))
    for c in g["cases"]:
        res = _run_case(c)
        got = [{"queue": b.queue, "reqs": b.reqs, "s": b.s, "P": b.P, "close": b.close_ns,
                "dispatch": b.dispatch_ns, "done": b.done_ns} for b in res.batches]
        assert got == c["batches"], c["name"]
        arr = np.array([r[0] for r in c["requests"]])
        assert res.latency_ns(arr).tolist() == c["latency"], c["name"]


# ------------------------------------------------------------- brute force

def _valid_groups(arr, n, B, T, end_t):
    """All order-preserving partitions of one queue's requests that obey the
    closing rules, stated declaratively; each with its close times."""
    m = len(arr)
    out = []
    for cuts in itertools.product([0, 1], repeat=max(m - 1, 0)):
        groups, cur = [], [0]
        for i in range(1, m):
            if cuts[i - 1]:
                groups.append(cur)
                cur = [i]
            else:
                cur.append(i)
        groups.append(cur)
        closes, ok = [], True
        for gi, g in enumerate(groups):
            o = arr[g[0]]
            s = sum(n[i] for i in g)
            if s > B:
                ok = False
                break
            # every member arrived strictly before the timeout
            if T is not None and arr[g[-1]] >= o + T:
                ok = False
                break
            if s == B:
                closes.append(arr[g[-1]])
                continue
            if gi + 1 < len(groups):
                nxt = groups[gi + 1][0]
                reasons = []
                if s + n[nxt] > B:
                    reasons.append(arr[nxt])          # the next request does not fit
                if T is not None and arr[nxt] >= o + T:
                    reasons.append(o + T)             # timed out before it came
                if not reasons:
                    ok = False                        # it would have joined this batch
                    break
                closes.append(min(reasons))
            else:
                closes.append(o + T if T is not None else end_t)
        if ok:
            out.append((groups, closes))
    return out


@pytest.mark.parametrize("seed", range(60))
def test_formation_matches_bruteforce(seed):
    rng = np.random.default_rng(seed)
    nq = int(rng.integers(1, 3))
    N = int(rng.integers(1, 8))
    qs = []
    for _ in range(nq):
        B = int(rng.integers(1, 6))
        T = None if rng.random() < 0.4 else int(rng.integers(1, 30))
        qs.append(ob.QueueCfg(B, (), T))
    arrival = np.sort(rng.integers(0, 40, size=N))
    rq = rng.integers(0, nq, size=N)
    n = np.array([int(rng.integers(1, qs[q].max_batch_size + 1)) for q in rq])
    svc = [[int(rng.integers(0, 20))] * (q.max_batch_size + 1) for q in qs]
    res = ob.simulate(qs, rq.tolist(), arrival.tolist(), n.tolist(), svc)
    for q in range(nq):
        idx = [i for i in range(N) if rq[i] == q]
        if not idx:
            continue
        valid = _valid_groups([int(arrival[i]) for i in idx], [int(n[i]) for i in idx],
                              qs[q].max_batch_size, qs[q].timeout_ns, int(arrival[-1]))
        assert len(valid) == 1, (seed, q, valid)
        groups, closes = valid[0]
        want = [([idx[i] for i in g], c) for g, c in zip(groups, closes)]
        mine = sorted([(b.reqs, b.close_ns) for b in res.batches if b.queue == q],
                      key=lambda x: x[0][0])
        assert mine == want, seed


@pytest.mark.parametrize("n,B,N", [(1, 8, 37), (2, 8, 50), (4, 16, 33), (8, 8, 5), (3, 12, 100)])
def test_equal_sizes_closed_form(n, B, N):
    qs = [ob.QueueCfg(B, (), None)]
    res = ob.simulate(qs, [0] * N, list(range(N)), [n] * N, [[1] * (B + 1)])
    assert len(res.batches) == math.ceil(N * n / B)
    assert all(b.s == B for b in res.batches[:-1])
    assert res.batches[-1].s == N * n - (len(res.batches) - 1) * B


def test_padded_size():
    assert ob.padded_size(1, (8, 16, 32)) == 8
    assert ob.padded_size(8, (8, 16, 32)) == 8
    assert ob.padded_size(9, (8, 16, 32)) == 16
    assert ob.padded_size(17, (8, 16, 32)) == 32
    assert ob.padded_size(13, ()) == 13
    with pytest.raises(ValueError):
        ob.padded_size(33, (8, 16, 32))


def test_bucket_choice():
    qs = [ob.QueueCfg(64, (), None, b) for b in (64, 128, 256, 512)]
    assert [ob.pick_queue(qs, [0, 1, 2, 3], L) for L in (1, 64, 65, 128, 129, 512)] == [0, 0, 1, 1, 2, 3]
    with pytest.raises(ValueError):
        ob.pick_queue(qs, [0, 1, 2, 3], 513)


# ------------------------------------------------------------- dispatch invariants

def _random_sim(seed, n_req=400):
    rng = np.random.default_rng(seed)
    nq = int(rng.integers(1, 6))
    qs = []
    for _ in range(nq):
        B = int(rng.integers(1, 40))
        allowed = ()
        if B > 1 and rng.random() < 0.5:
            allowed = tuple(sorted(set(int(x) for x in rng.integers(1, B, size=3)) | {B}))
        T = None if rng.random() < 0.3 else int(rng.integers(1, 500))
        qs.append(ob.QueueCfg(B, allowed, T))
    arrival = np.cumsum(rng.integers(0, 30, size=n_req))
    rq = rng.integers(0, nq, size=n_req)
    n = np.array([int(rng.integers(1, qs[q].max_batch_size + 1)) for q in rq])
    svc = [[int(rng.integers(1, 200)) for _ in range(q.max_batch_size + 1)] for q in qs]
    return qs, rq, arrival, n, svc, ob.simulate(qs, rq.tolist(), arrival.tolist(), n.tolist(), svc)


@pytest.mark.parametrize("seed", range(25))
def test_dispatch_log_invariants(seed):
    qs, rq, arrival, n, svc, res = _random_sim(seed)
    nq = len(qs)
    seen = np.zeros(len(arrival), dtype=int)
    remaining = list(res.batches)
    prev_done, last = None, -1
    for i, b in enumerate(res.batches):
        # every batch holds its queue's requests in arrival order, within limits
        assert all(rq[r] == b.queue for r in b.reqs)
        assert b.reqs == sorted(b.reqs)
        assert b.s == sum(n[r] for r in b.reqs) <= qs[b.queue].max_batch_size
        assert b.P == ob.padded_size(b.s, qs[b.queue].allowed)
        seen[b.reqs] += 1
        assert b.dispatch_ns >= b.close_ns >= arrival[b.reqs[-1]]
        assert b.done_ns == b.dispatch_ns + svc[b.queue][b.P]
        # serial and work-conserving: it starts when the device frees up or,
        # if nothing was waiting then, at the next close
        rest = remaining[i:]
        earliest = min(x.close_ns for x in rest)
        want = earliest if prev_done is None else max(prev_done, earliest)
        assert b.dispatch_ns == want
        # round robin: first queue after the last-served one with a closed batch
        ready = {x.queue for x in rest if x.close_ns <= b.dispatch_ns}
        cyc = [(last + k) % nq for k in range(1, nq + 1)]
        assert b.queue == next(q for q in cyc if q in ready)
        # FIFO within the queue
        assert b.close_ns == min(x.close_ns for x in rest if x.queue == b.queue)
        prev_done, last = b.done_ns, b.queue
    assert np.all(seen == 1)


@pytest.mark.parametrize("seed", range(10))
def test_littles_law_sample_path(seed):
    qs, rq, arrival, n, svc, res = _random_sim(seed, n_req=300)
    lat = res.latency_ns(arrival)
    assert np.all(lat >= 0)
    # integral of the number of requests in the system, by an event sweep
    ev = sorted([(int(a), 1) for a in arrival] + [(int(d), -1) for d in res.done_ns])
    area, cnt, t_prev = 0, 0, ev[0][0]
    for t, d in ev:
        area += cnt * (t - t_prev)
        cnt += d
        t_prev = t
    assert cnt == 0
    assert int(lat.sum()) == area


def _random_windowed(seed, n_req=400):
    rng = np.random.default_rng(7000 + seed)
    qs, rq, arrival, n, svc, _ = _random_sim(seed, n_req)
    W = int(rng.integers(2, 7))
    wns = [int(rng.integers(0, 300)) for _ in qs]
    tails = [int(rng.integers(0, 500)) if seed % 2 else 0 for _ in qs]
    res = ob.simulate(qs, rq.tolist(), arrival.tolist(), n.tolist(), svc, W, wns, tails)
    return qs, rq, arrival, n, svc, W, (wns, tails), res


@pytest.mark.parametrize("seed", range(25))
def test_launch_window_invariants(seed):
    # the windowed device restated declaratively from the batches' close
    # times alone: each window starts when the device frees up (or at the
    # next close when nothing waits), takes min(W, waiting) batches in
    # round-robin order (FIFO within a queue), holds the device for the sum
    # of its queues' chain times and its batches' service times, and its
    # batches complete its queues' tails after that
    qs, rq, arrival, n, svc, W, (wns, tails), res = _random_windowed(seed)
    nq = len(qs)
    wins = []
    for b in res.batches:
        if not wins or b.window != wins[-1][0].window:
            wins.append([])
        wins[-1].append(b)
    assert [w[0].window for w in wins] == list(range(len(wins)))
    done_prev, last, k = None, -1, 0
    for w in wins:
        rest = res.batches[k:]
        t = w[0].dispatch_ns
        earliest = min(x.close_ns for x in rest)
        assert t == (earliest if done_prev is None else max(done_prev, earliest))
        waiting = [x for x in rest if x.close_ns <= t]
        assert len(w) == min(W, len(waiting))
        picked = []
        for b in w:
            avail = [x for x in waiting if x not in picked]
            cyc = [(last + j) % nq for j in range(1, nq + 1)]
            q = next(q for q in cyc if any(x.queue == q for x in avail))
            assert b.queue == q
            assert b.close_ns == min(x.close_ns for x in avail if x.queue == q)
            picked.append(b)
            last = q
        busy = sum(wns[q] for q in {b.queue for b in w}) + sum(svc[b.queue][b.P] for b in w)
        tail = sum(tails[q] for q in {b.queue for b in w})
        assert all(b.dispatch_ns == t and b.done_ns == t + busy + tail for b in w)
        done_prev = t + busy
        k += len(w)
    assert sorted(r for b in res.batches for r in b.reqs) == list(range(len(arrival)))


@pytest.mark.parametrize("seed", range(10))
def test_window_of_one_adds_chain_time_to_service(seed):
    # W = 1 with chain times a_q is the one-batch device with service S + a_q
    qs, rq, arrival, n, svc, W, (wns, _), _ = _random_windowed(seed)
    r1 = ob.simulate(qs, rq.tolist(), arrival.tolist(), n.tolist(), svc, 1, wns)
    svc2 = [[s + wns[q] for s in row] for q, row in enumerate(svc)]
    r2 = ob.simulate(qs, rq.tolist(), arrival.tolist(), n.tolist(), svc2)
    key = lambda r: [(b.queue, b.reqs, b.s, b.P, b.close_ns, b.dispatch_ns, b.done_ns) for b in r.batches]
    assert key(r1) == key(r2)
    assert np.array_equal(r1.done_ns, r2.done_ns)


@pytest.mark.parametrize("seed", range(5))
def test_littles_law_with_windows(seed):
    qs, rq, arrival, n, svc, W, _, res = _random_windowed(seed, n_req=300)
    lat = res.latency_ns(arrival)
    ev = sorted([(int(a), 1) for a in arrival] + [(int(d), -1) for d in res.done_ns])
    area, cnt, t_prev = 0, 0, ev[0][0]
    for t, d in ev:
        area += cnt * (t - t_prev)
        cnt += d
        t_prev = t
    assert cnt == 0 and int(lat.sum()) == area


def test_composition_independent_of_service_times():
    qs, rq, arrival, n, svc, res = _random_sim(3)
    svc2 = [[s * 7 + 3 for s in row] for row in svc]
    res2 = ob.simulate(qs, rq.tolist(), arrival.tolist(), n.tolist(), svc2)
    key = lambda r: sorted((b.queue, tuple(b.reqs), b.s, b.P, b.close_ns) for b in r.batches)
    assert key(res) == key(res2)


def test_dst_rows_and_percentiles():
    assert ob.dst_rows([3, 1, 4, 1]).tolist() == [0, 3, 4, 8]
    assert ob.dst_rows([]).tolist() == []
    v = [50, 10, 40, 20, 30]
    assert ob.percentile_nearest_rank(v, 0.5) == 30     # ceil(2.5) = 3rd smallest
    assert ob.percentile_nearest_rank(v, 0.99) == 50
    assert ob.percentile_nearest_rank(list(range(1, 101)), 0.99) == 99
    assert ob.percentile_nearest_rank(list(range(1, 101)), 0.5) == 50
