"""The C ABI without a GPU: the library loads and exports every entry point
include/rb.h declares; status codes and ownership rules on the host paths
(host-only context, no-device scheduler); the serving API's batch formation
against the oracle."""
import os
import re

import numpy as np
import pytest

from oracle import batching as ob
from paper_1712_06139_amd import rb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "rb.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^(?:rb_status|const char\*)\s+(rb_[a-z0-9_]+)\s*\(", src, flags=re.M)))


def test_every_declared_symbol_is_exported_and_bound():
    names = declared_functions()
    assert len(names) >= 28
    lib = rb.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(rb.EXPORTS) == names


def test_every_declared_call_cites_its_passage():
    # each exported call's own comment block names the paper section that
    # defines the operation
    src = open(os.path.join(ROOT, "include", "rb.h")).read()
    decl = re.compile(r"^(?:rb_status|const char\*)\s+(rb_\w+)\(", re.M)
    names = []
    prev_end = 0
    for m in decl.finditer(src):
        block = src[prev_end:m.start()]
        comments = re.findall(r"/\*.*?\*/", block, re.S)
        assert comments, m.group(1)
        text = re.sub(r"\s*\n\s*\*?\s*", " ", comments[-1])
        # the allocation-free variant names the callers it is for instead
        assert re.search(r"section \d+(\.\d+)*", text) or "cannot allocate" in text, m.group(1)
        names.append(m.group(1))
        prev_end = src.index(";", m.end()) + 1
    assert set(names) == set(rb.EXPORTS)


def test_status_strings():
    for code in (rb.RB_OK, rb.RB_EINVAL, rb.RB_EBUSY, rb.RB_EAGAIN, rb.RB_EEMPTY, rb.RB_ESIZE, rb.RB_ENOENT,
                 rb.RB_EDEVICE, rb.RB_ENOMEM, rb.RB_ERANGE):
        assert rb.lib().rb_status_str(code)
    assert rb.lib().rb_status_str(-1234) == b"unknown status"


@pytest.fixture
def ctx():
    c = rb.Ctx(-1)
    yield c


def mlp(ctx, d_in=4, d_out=3):
    return rb.Model(ctx, "mlp", "f32", [(None, None, "relu"), (None, None, "none")],
                    shapes=[(8, d_in), (d_out, 8)])


def status(fn):
    try:
        fn()
    except rb.RBError as e:
        return e.status
    return rb.RB_OK


def test_model_validation(ctx):
    # layer chain mismatch
    assert status(lambda: rb.Model(ctx, "mlp", "f32", [(None, None, "relu"), (None, None, "none")],
                                   shapes=[(8, 4), (3, 9)])) == rb.RB_EINVAL
    # softmax is not a layer activation
    assert status(lambda: rb.Model(ctx, "mlp", "f32", [(None, None, "softmax")], shapes=[(3, 4)])) == rb.RB_EINVAL
    # ranking: first layer must take n_tables * 64 + n_dense inputs
    assert status(lambda: rb.Model(ctx, "ranking", "bf16", [(None, None, "sigmoid")], n_dense=13,
                                   shapes=[(1, 26 * 64 + 12), (26, 0)], table_rows=10)) == rb.RB_EINVAL
    # a device context needs weights
    m = mlp(ctx)
    assert (m.d_in, m.d_out) == (4, 3)
    m.destroy()


def test_queue_validation(ctx):
    s = rb.Sched(ctx, device=False)
    m = mlp(ctx)
    bad = [dict(max_batch_size=0), dict(max_batch_size=8, allowed=(4, 2, 8)), dict(max_batch_size=8, allowed=(2, 4)),
           dict(max_batch_size=8, allowed=(2, 2, 8)), dict(max_batch_size=8, timeout_ns=0),
           dict(max_batch_size=5000), dict(max_batch_size=8, bucket_len=64),
           dict(max_batch_size=8, service_ns=[1, 2, 3])]
    for kw in bad:
        kw = dict(kw)
        B = kw.pop("max_batch_size")
        assert status(lambda: rb.Queue(s, m, B, **kw)) == rb.RB_EINVAL, kw
    q = rb.Queue(s, m, 8, (2, 4, 8), None, 0, list(range(9)))
    q.destroy()
    s.destroy()
    m.destroy()


def test_device_mode_needs_a_device(ctx):
    assert status(lambda: rb.Sched(ctx, device=True)) == rb.RB_EDEVICE


def test_stream_count_bounds(ctx):
    assert status(lambda: rb.Sched(ctx, device=False, n_streams=-1)) == rb.RB_EINVAL
    assert status(lambda: rb.Sched(ctx, device=False, n_streams=17)) == rb.RB_EINVAL
    rb.Sched(ctx, device=False, n_streams=16).destroy()
    assert status(lambda: rb.Sched(ctx, device=False, seq_pack=2)) == rb.RB_EINVAL
    assert status(lambda: rb.Sched(ctx, device=False, seq_pack=-1)) == rb.RB_EINVAL
    rb.Sched(ctx, device=False, seq_pack=True).destroy()
    assert status(lambda: rb.Sched(ctx, device=False, profile=3)) == rb.RB_EINVAL
    assert status(lambda: rb.Sched(ctx, device=False, profile=-1)) == rb.RB_EINVAL


def test_ownership_and_busy_rules(ctx):
    s = rb.Sched(ctx, device=False)
    m = mlp(ctx)
    q = rb.Queue(s, m, 8, (), None)
    x = np.zeros((2, 4), np.float32)
    # oversize request, wrong payload size, time going backwards
    assert status(lambda: s.submit(q, 9, np.zeros((9, 4), np.float32), arrival_ns=0)) == rb.RB_EINVAL
    assert status(lambda: s.submit(q, 2, np.zeros(7, np.float32), arrival_ns=0)) == rb.RB_EINVAL
    rid = s.submit(q, 2, x, arrival_ns=100)
    assert status(lambda: s.submit(q, 2, x, arrival_ns=50)) == rb.RB_EINVAL
    assert status(lambda: s.advance(10)) == rb.RB_EINVAL
    # pending work keeps queue, model, scheduler and context alive
    assert status(q.destroy) == rb.RB_EBUSY
    assert status(m.destroy) == rb.RB_EBUSY
    assert status(s.destroy) == rb.RB_EBUSY
    assert status(ctx.destroy) == rb.RB_EBUSY
    # not run yet -> not ready; unknown -> no entry
    assert status(lambda: s.collect(rid, 2, 3)) == rb.RB_EAGAIN
    assert status(lambda: s.collect(rid + 10, 2, 3)) == rb.RB_ENOENT
    assert s.run_next() is None          # the open batch is not closed yet
    rb.check(rb.lib().rb_flush(q.h), "rb_flush")
    b = s.run_next()
    assert b["reqs"] == [rid] and b["real"] == 2 and b["padded"] == 2
    assert s.run_next() is None
    # no device: there are no outputs to collect
    assert status(lambda: s.collect(rid, 2, 3)) == rb.RB_EDEVICE
    q.destroy()
    m.destroy()
    s.destroy()


def test_version_transition_rules(ctx):
    # a queue switches to a new version of the same shape; the old version is
    # then unbound (destroyable) and the new one bound (busy)
    s = rb.Sched(ctx, device=False)
    old, new, other = mlp(ctx), mlp(ctx), mlp(ctx, d_in=5)
    q1 = rb.Queue(s, old, 8, (), None)
    q2 = rb.Queue(s, old, 8, (), None)
    assert status(lambda: q1.set_model(other)) == rb.RB_EINVAL   # different input width
    assert status(lambda: rb.check(rb.lib().rb_queue_set_model(None, new.h), "x")) == rb.RB_EINVAL
    q1.set_model(new)
    assert status(old.destroy) == rb.RB_EBUSY      # q2 still serves the old version
    rid = s.submit(q1, 2, np.zeros((2, 4), np.float32), arrival_ns=0)
    q2.set_model(new)
    old.destroy()
    assert status(new.destroy) == rb.RB_EBUSY
    rb.check(rb.lib().rb_flush(q1.h), "rb_flush")
    assert s.run_next()["reqs"] == [rid]
    q1.set_model(new)                              # same model: no-op
    q1.destroy()
    q2.destroy()
    new.destroy()
    other.destroy()
    s.destroy()


def test_resource_preserving_transition(ctx):
    # the queue is held (no version bound): the old version can be destroyed
    # before the new one exists; requests keep arriving and batches keep
    # closing, but nothing is dispatched until a version is set again
    s = rb.Sched(ctx, device=False)
    old, other = mlp(ctx), mlp(ctx, d_out=5)
    q = rb.Queue(s, old, 8, (), None)
    q2 = rb.Queue(s, mlp(ctx), 8, (), None)
    r1 = s.submit(q, 2, np.zeros((2, 4), np.float32), arrival_ns=0)
    rb.check(rb.lib().rb_flush(q.h), "rb_flush")
    q.set_model(None)
    old.destroy()                                   # nothing serves it any more
    r2 = s.submit(q, 3, np.zeros((3, 4), np.float32), arrival_ns=10)
    assert status(lambda: s.submit(q, 1, np.zeros((1, 5), np.float32), arrival_ns=10)) == rb.RB_EINVAL
    rb.check(rb.lib().rb_flush(q.h), "rb_flush")
    r3 = s.submit(q2, 1, np.zeros((1, 4), np.float32), arrival_ns=20)
    rb.check(rb.lib().rb_flush(q2.h), "rb_flush")
    assert s.run_next()["reqs"] == [r3]             # other queues keep being served
    assert s.run_next() is None                     # the held queue dispatches nothing
    m3 = mlp(ctx)
    q3 = rb.Queue(s, m3, 8, (), None)
    q3.set_model(None)                              # held and empty: a replay could not drain it
    assert status(lambda: s.sim_run([[q3]], np.zeros(1), np.zeros(1), np.ones(1))) == rb.RB_EBUSY
    q3.destroy()
    m3.destroy()
    assert status(lambda: q.set_model(other)) == rb.RB_EINVAL   # different output width
    new = mlp(ctx)
    q.set_model(new)
    assert s.run_next()["reqs"] == [r1]
    assert s.run_next()["reqs"] == [r2]
    assert s.run_next() is None
    q.destroy()
    q2.model_ = q2.model
    q2.destroy()
    for m in (new, other, q2.model_):
        m.destroy()
    s.destroy()


def test_sim_run_argument_checks(ctx):
    s = rb.Sched(ctx, device=False)
    m = mlp(ctx)
    q = rb.Queue(s, m, 8, (), None)
    n_rows = np.array([1, 2, 3])
    arr = np.array([0, 5, 3])
    assert status(lambda: s.sim_run([[q]], np.zeros(3), arr, n_rows)) == rb.RB_EINVAL   # time goes back
    assert status(lambda: s.sim_run([[q]], np.array([0, 1, 0]), np.sort(arr), n_rows)) == rb.RB_EINVAL
    assert status(lambda: s.sim_run([[q]], np.zeros(3), np.sort(arr), np.array([1, 9, 1]))) == rb.RB_EINVAL
    # a queue that still holds requests cannot take part in a replay
    s.submit(q, 1, np.zeros((1, 4), np.float32), arrival_ns=0)
    assert status(lambda: s.sim_run([[q]], np.zeros(3), np.sort(arr), n_rows)) == rb.RB_EBUSY
    rb.check(rb.lib().rb_flush(q.h), "rb_flush")
    s.run_next()
    log = s.sim_run([[q]], np.zeros(3), np.sort(arr), n_rows)
    assert log["n_batches"] == 1 and log["b_real"].tolist() == [6]
    q.destroy()
    m.destroy()
    s.destroy()


@pytest.mark.parametrize("seed", range(12))
def test_serving_api_formation_matches_oracle(ctx, seed):
    # submit / advance / flush / run_next or run_window on several queues with
    # timeouts, service tables, chain times and launch windows: the batches
    # (composition, close, dispatch and done times, windows) equal the
    # oracle's on the same arrivals. Arrivals of one timestamp are submitted
    # before the batches are run; count-only queues are flushed after the last
    # arrival (the end-of-trace close)
    rng = np.random.default_rng(seed)
    nq = int(rng.integers(1, 4))
    W = 1 if seed % 3 == 0 else int(rng.integers(2, 6))
    use_window = seed % 2 == 1
    cfg = []
    for _ in range(nq):
        B = int(rng.integers(2, 20))
        T = None if rng.random() < 0.3 else int(rng.integers(5, 100))
        cfg.append(ob.QueueCfg(B, (), T))
    svc = [[int(rng.integers(0, 40)) for _ in range(c.max_batch_size + 1)] for c in cfg]
    wns = [int(rng.integers(0, 30)) for _ in range(nq)]
    tails = [int(rng.integers(0, 60)) for _ in range(nq)]
    N = 300
    arrival = np.cumsum(rng.integers(0, 20, size=N))
    rq = rng.integers(0, nq, size=N)
    n = np.array([int(rng.integers(1, cfg[q].max_batch_size + 1)) for q in rq])
    s = rb.Sched(ctx, device=False, window_batches=W)
    m = mlp(ctx)
    qs = [rb.Queue(s, m, c.max_batch_size, (), c.timeout_ns, 0, svc[i], wns[i], tails[i])
          for i, c in enumerate(cfg)]
    got = []

    def drain():
        while True:
            if use_window:
                win = s.run_window()
                if win is None:
                    return
                assert 1 <= len(win) <= W
                assert len({(b["dispatch_ns"], b["done_ns"]) for b in win}) == 1
                batches = win
            else:
                b = s.run_next()
                if b is None:
                    return
                batches = [b]
            for b in batches:
                got.append((b["queue"], b["reqs"], b["close_ns"], b["dispatch_ns"], b["done_ns"]))

    r = 0
    while r < N:
        t = int(arrival[r])
        while r < N and arrival[r] == t:
            s.submit(qs[rq[r]], int(n[r]), np.zeros((int(n[r]), 4), np.float32), arrival_ns=t)
            r += 1
        if r == N:
            for q, c in zip(qs, cfg):
                if c.timeout_ns is None:
                    rb.check(rb.lib().rb_flush(q.h), "rb_flush")
        drain()
    s.advance(int(arrival[-1]) + 10 ** 12)   # past every timeout and the device's backlog
    drain()
    ref = ob.simulate(cfg, rq.tolist(), arrival.tolist(), n.tolist(), svc, W, wns, tails)
    assert got == [(b.queue, list(b.reqs), b.close_ns, b.dispatch_ns, b.done_ns) for b in ref.batches]
    for q in qs:
        q.destroy()
    m.destroy()
    s.destroy()


def test_replay_refuses_a_scheduler_with_waiting_requests(ctx):
    # a replay runs the scheduler's clock over all of its queues: a closed
    # batch waiting on a queue outside the replay, served or held, makes the
    # replay refuse (instead of serving it as part of the replay, or waiting
    # forever for a held queue)
    s = rb.Sched(ctx, device=False)
    m1, m2 = mlp(ctx), mlp(ctx)
    q1 = rb.Queue(s, m1, 8, (), None)
    q2 = rb.Queue(s, m2, 8, (), None)
    args = ([[q1]], np.zeros(2), np.array([0, 1]), np.array([1, 2]))
    s.submit(q2, 2, np.zeros((2, 4), np.float32), arrival_ns=0)
    rb.check(rb.lib().rb_flush(q2.h), "rb_flush")
    assert status(lambda: s.sim_run(*args)) == rb.RB_EBUSY
    assert s.run_next()["queue"] == q2.id
    s.submit(q2, 1, np.zeros((1, 4), np.float32), arrival_ns=5)
    rb.check(rb.lib().rb_flush(q2.h), "rb_flush")
    q2.set_model(None)
    assert status(lambda: s.sim_run(*args)) == rb.RB_EBUSY
    q2.set_model(m2)
    assert s.run_next()["queue"] == q2.id
    log = s.sim_run(*args)
    assert log["n_batches"] == 1 and log["b_reqs"].tolist() == [0, 1]
    for o in (q1, q2, m1, m2, s):
        o.destroy()
