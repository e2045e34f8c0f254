"""Host logic of the library against the oracle, without a GPU: the
no-device scheduler replays every workload's full trace and must produce
the oracle's batch log bit for bit (composition, padded sizes, dispatch order
and simulated times), and the hand-worked schedules."""
import json
import os

import numpy as np
import pytest

import synth
from oracle import batching as ob
from paper_1712_06139_amd import rb
from paper_1712_06139_amd.deploy import Deployment

from helpers import lib_batches, oracle_batches, oracle_sim, service_table


@pytest.fixture(scope="module")
def ctx():
    c = rb.Ctx(-1)
    yield c


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
@pytest.mark.parametrize("window", [1, 64])
def test_full_trace_log_matches_oracle(ctx, name, window):
    w = synth.workload(name)
    t = synth.trace(w)
    svc = service_table(w)
    wns = [3_000 + 1_000 * i for i in range(len(w.queues))]
    tails = [0 if window == 1 else 50_000 + 7_000 * i for i in range(len(w.queues))]
    dep = Deployment(w, ctx, device=False, service_ns=svc, with_params=False, window_batches=window,
                     window_ns=wns, window_tail_ns=tails)
    try:
        log = dep.replay_meta(t)
        ours = lib_batches(log, dep.qindex)
        ref = oracle_sim(w, t, svc, window, wns, tails)
        assert ours == oracle_batches(ref)
        assert np.array_equal(log["req_done_ns"], ref.done_ns)
        # a second replay on the same scheduler starts a fresh clock
        log2 = dep.replay_meta(t)
        assert lib_batches(log2, dep.qindex) == ours
    finally:
        dep.destroy()


def test_hand_worked_schedules_through_library(ctx, golden_dir):
    g = json.load(open(os.path.join(golden_dir, "schedule_cases.json")))
    for c in g["cases"]:
        sched = rb.Sched(ctx, device=False, window_batches=c.get("window", 1))
        m = rb.Model(ctx, "mlp", "f32", [(None, None, "none")], shapes=[(4, 4)])
        wns = c.get("window_ns", [0] * len(c["queues"]))
        tails = c.get("window_tail_ns", [0] * len(c["queues"]))
        qs = [rb.Queue(sched, m, q["max_batch_size"], q["allowed"], q["timeout_ns"], 0, c["service_ns"][i], wns[i],
                       tails[i])
              for i, q in enumerate(c["queues"])]
        req = c["requests"]
        log = sched.sim_run([[q] for q in qs], np.array([r[1] for r in req]), np.array([r[0] for r in req]),
                            np.array([r[2] for r in req]))
        got = [{"queue": q, "reqs": reqs, "s": s, "P": P, "close": cl, "dispatch": di, "done": do}
               for (q, reqs, s, P, cl, di, do) in lib_batches(log, {q.id: i for i, q in enumerate(qs)})]
        assert got == c["batches"], c["name"]
        for q in qs:
            q.destroy()
        sched.destroy()
        m.destroy()


@pytest.mark.parametrize("seed", range(20))
def test_random_traces_match_oracle(ctx, seed):
    rng = np.random.default_rng(100 + seed)
    nq = int(rng.integers(1, 6))
    cfg = []
    for _ in range(nq):
        B = int(rng.integers(1, 40))
        allowed = ()
        if B > 1 and rng.random() < 0.5:
            allowed = tuple(sorted(set(int(x) for x in rng.integers(1, B, size=3)) | {B}))
        T = None if rng.random() < 0.3 else int(rng.integers(1, 500))
        cfg.append(ob.QueueCfg(B, allowed, T))
    N = 500
    arrival = np.cumsum(rng.integers(0, 30, size=N))
    rq = rng.integers(0, nq, size=N)
    n = np.array([int(rng.integers(1, cfg[q].max_batch_size + 1)) for q in rq])
    svc = [[int(rng.integers(0, 200)) for _ in range(c.max_batch_size + 1)] for c in cfg]
    W = 1 if seed < 10 else int(rng.integers(2, 9))
    wns = [0] * nq if seed < 10 else [int(rng.integers(0, 300)) for _ in range(nq)]
    tails = [0] * nq if seed < 15 else [int(rng.integers(0, 900)) for _ in range(nq)]
    ref = ob.simulate(cfg, rq.tolist(), arrival.tolist(), n.tolist(), svc, W, wns, tails)
    sched = rb.Sched(ctx, device=False, window_batches=W)
    m = rb.Model(ctx, "mlp", "f32", [(None, None, "none")], shapes=[(4, 4)])
    qs = [rb.Queue(sched, m, c.max_batch_size, c.allowed, c.timeout_ns, 0, svc[i], wns[i], tails[i])
          for i, c in enumerate(cfg)]
    log = sched.sim_run([[q] for q in qs], rq, arrival, n)
    assert lib_batches(log, {q.id: i for i, q in enumerate(qs)}) == oracle_batches(ref)
    for q in qs:
        q.destroy()
    sched.destroy()
    m.destroy()
