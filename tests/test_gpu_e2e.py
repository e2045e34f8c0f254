"""End-to-end GPU parity: every workload's trace (a prefix sized for the
oracle) is replayed through the library on the GPU; the batch log must equal
the oracle's bit for bit and every request's output rows must match the
oracle's unbatched forward of that request within the tolerance of its
precision (row-scaled: max_j |y_j - ref_j| <= rtol * max_j |ref_j|, rtol 1e-5
for fp32 models, 2e-2 for bf16 weights with fp32 accumulation). Also: NaN
padding never reaches an output, outputs do not depend on the launch window
(bit for bit), and the serving API (submit / run_next / collect)."""
import functools

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth
from oracle.models import OracleModel
from paper_1712_06139_amd import rb
from paper_1712_06139_amd.deploy import Deployment

from helpers import group_descriptors, lib_batches, oracle_batches, oracle_sim, service_table

pytestmark = pytest.mark.gpu

RTOL = {"f32": 1e-5, "bf16": 2e-2}

PREFIX = {"small_mlp": 256, "ranking": 1200, "large_mlp": 72, "multi_tenant": 1500, "ragged_seq": 300}


@pytest.fixture(scope="module")
def ctx():
    c = rb.Ctx(0)
    yield c


@functools.lru_cache(maxsize=None)
def oracle_model(name, s):
    w = synth.workload(name)
    return OracleModel(w.models[s], synth.model_params(w, s))


@functools.lru_cache(maxsize=None)
def trace_and_arenas(name, n):
    w = synth.workload(name)
    t = synth.trace(w, n)
    return t, synth.arenas(t)


def row_scaled_err(y, ref):
    scale = np.maximum(np.max(np.abs(ref), axis=1, keepdims=True), 1e-30)
    return float(np.max(np.abs(y.astype(np.float64) - ref) / scale))


def run(ctx, name, n, window=1, pad=0.0, profile=False, n_streams=1, seq_pack=False, emb_dedup=False,
        fused_tail=False):
    w = synth.workload(name)
    t, a = trace_and_arenas(name, n)
    svc = service_table(w)
    dep = Deployment(w, ctx, device=True, window_batches=window, pad_value=pad, service_ns=svc, profile=profile,
                     n_streams=n_streams, seq_pack=seq_pack, emb_dedup=emb_dedup, fused_tail=fused_tail)
    try:
        dt = dep.upload(t, a)
        log = dep.replay(dt)
        dep.sched.sync()
        out = dt.out.cpu().numpy()
        return w, t, a, dep.qindex, log, out, dt.out_off
    finally:
        dep.destroy()


def check_outputs(name, t, a, out, out_off, reqs):
    w = synth.workload(name)
    worst = 0.0
    for r in reqs:
        s = int(t.servable[r])
        om = oracle_model(name, s)
        ref = om.forward(a.payload(r))
        y = out[out_off[r]:out_off[r + 1]].reshape(ref.shape)
        assert np.isfinite(y).all(), r
        e = row_scaled_err(y, ref.astype(np.float64))
        worst = max(worst, e)
        assert e <= RTOL[w.models[s].dtype], (name, r, e)
    return worst


@pytest.mark.parametrize("name", list(PREFIX))
def test_workload_prefix_matches_oracle(ctx, name):
    n = PREFIX[name]
    w, t, a, qindex, log, out, out_off = run(ctx, name, n)
    assert lib_batches(log, qindex) == oracle_batches(oracle_sim(w, t, service_table(w)))
    worst = check_outputs(name, t, a, out, out_off, range(t.n))
    print(f"{name}: {t.n} requests, worst row-scaled error {worst:.3g}")


@pytest.mark.parametrize("name", ["small_mlp", "ranking", "ragged_seq"])
def test_nan_padding_never_leaks(ctx, name):
    n = min(PREFIX[name], 400)
    *_, out0, _ = run(ctx, name, n, pad=0.0)
    *_, out1, _ = run(ctx, name, n, pad=float("nan"))
    assert np.isfinite(out1).all()
    assert np.array_equal(out0, out1)


@pytest.mark.parametrize("name", ["small_mlp", "ranking", "large_mlp", "ragged_seq"])
def test_outputs_independent_of_launch_window(ctx, name):
    n = min(PREFIX[name], 600)
    *_, out1, _ = run(ctx, name, n, window=1)
    *_, out8, _ = run(ctx, name, n, window=8)
    assert np.array_equal(out1, out8)


@pytest.mark.parametrize("name,n_streams", [("multi_tenant", 4), ("multi_tenant", 3), ("ragged_seq", 4),
                                            ("ranking", 2)])
def test_outputs_independent_of_stream_count(ctx, name, n_streams):
    # concurrent launch chains of different models, and consecutive chains of
    # one model alternating between two work-buffer slots on two lanes
    # (ranking: one model; ragged_seq: one model over four bucket queues),
    # change nothing
    n = min(PREFIX[name], 1500)
    w, t, a, qindex, log1, out1, _ = run(ctx, name, n, window=16)
    _, _, _, _, logk, outk, out_off = run(ctx, name, n, window=16, n_streams=n_streams)
    assert lib_batches(log1, qindex) == lib_batches(logk, qindex)
    assert np.array_equal(out1, outk)
    check_outputs(name, t, a, outk, out_off, range(0, t.n, 7))


def test_single_group_chunks_and_lanes_share_work_buffers(ctx):
    # with lanes, a replay chunk of one launch group runs on the scheduler's
    # own stream while chunks of several groups run on the lanes, with the same
    # work buffers: replays of both kinds enqueued back to back with no sync in
    # between give the same bits as one stream
    name = "ranking"
    n = min(PREFIX[name], 600)
    w, t, a, qindex, log1, out1, _ = run(ctx, name, n, window=16)
    t, a = trace_and_arenas(name, n)
    dep = Deployment(w, ctx, device=True, window_batches=16, service_ns=service_table(w), n_streams=8)
    try:
        dt = dep.upload(t, a)
        k = 1
        while k < n and int(t.n_rows[:k + 1].sum()) <= 512:
            k += 1

        def prefix(k):
            return dep.sched.sim_run(dep.servables, t.servable[:k], t.arrival_ns[:k], t.n_rows[:k], None,
                                     dense=dt.dense, dense_off=a.dense_off[:k + 1], lens=dt.lens,
                                     lens_off=a.lens_off[:k + 1], ids=dt.ids, ids_off=a.ids_off[:k + 1],
                                     out=dt.out, out_off=dt.out_off[:k + 1])
        logs = []
        for _ in range(3):
            logs.append(dep.replay(dt))
            assert int(prefix(k)["n_batches"]) == 1
        logs.append(dep.replay(dt))
        dep.sched.sync()
        out8 = dt.out.cpu().numpy()
    finally:
        dep.destroy()
    assert all(lib_batches(lg, qindex) == lib_batches(log1, qindex) for lg in logs)
    assert np.array_equal(out1, out8)


@pytest.mark.parametrize("name,window", [("ranking", 8), ("multi_tenant", 16)])
def test_embedding_dedup_bit_identical(ctx, name, window):
    # ranking models with each block's distinct table rows gathered once:
    # the same batches and the same output bits, with NaN padding too
    n = min(PREFIX[name], 1500)
    w, t, a, qindex, log0, out0, out_off = run(ctx, name, n, window=window)
    _, _, _, _, log1, out1, _ = run(ctx, name, n, window=window, emb_dedup=True)
    *_, out2, _ = run(ctx, name, n, window=window, emb_dedup=True, pad=float("nan"))
    assert lib_batches(log0, qindex) == lib_batches(log1, qindex)
    assert np.array_equal(out0, out1) and np.array_equal(out0, out2)


@pytest.mark.parametrize("name,window", [("ranking", 1), ("ranking", 16), ("multi_tenant", 16)])
def test_fused_mlp_tail_bit_identical(ctx, name, window):
    # the ranking MLP's last two layers and head in one kernel or three: the
    # same batches and the same output bits
    n = min(PREFIX[name], 1500)
    w, t, a, qindex, log0, out0, out_off = run(ctx, name, n, window=window)
    _, _, _, _, log1, out1, _ = run(ctx, name, n, window=window, fused_tail=True)
    assert lib_batches(log0, qindex) == lib_batches(log1, qindex)
    assert np.array_equal(out0, out1)


@pytest.mark.parametrize("window,pad", [(1, 0.0), (16, float("nan"))])
def test_packed_tokens_match_padded(ctx, window, pad):
    # sub-graph batching of the token-wise layers (real tokens packed, no time
    # padding): same batches, outputs bit-identical to the padded path, so
    # within the oracle's tolerance too
    name = "ragged_seq"
    n = min(PREFIX[name], 1500)
    w, t, a, qindex, log0, out0, out_off = run(ctx, name, n, window=window)
    _, _, _, _, log1, out1, _ = run(ctx, name, n, window=window, pad=pad, seq_pack=True)
    assert lib_batches(log0, qindex) == lib_batches(log1, qindex)
    assert np.isfinite(out1).all()
    assert np.array_equal(out0, out1)
    check_outputs(name, t, a, out1, out_off, range(0, t.n, 5))


def test_serving_api_matches_oracle(ctx):
    name = "small_mlp"
    w = synth.workload(name)
    t, a = trace_and_arenas(name, 256)
    dep = Deployment(w, ctx, device=True, service_ns=service_table(w))
    try:
        q = dep.queues[0]
        ids = []
        for r in range(t.n):
            p = a.payload(r)
            ids.append(dep.sched.submit(q, int(t.n_rows[r]), p.dense, arrival_ns=int(t.arrival_ns[r])))
            while dep.sched.run_next() is not None:
                pass
        rb.check(rb.lib().rb_flush(q.h), "rb_flush")
        while dep.sched.run_next() is not None:
            pass
        dep.sched.sync()
        om = oracle_model(name, 0)
        for r in range(t.n):
            y = dep.sched.collect(ids[r], int(t.n_rows[r]), 16)
            ref = om.forward(a.payload(r))
            assert row_scaled_err(y, ref.astype(np.float64)) <= RTOL["f32"]
        with pytest.raises(rb.RBError) as e:
            dep.sched.collect(ids[0], int(t.n_rows[0]), 16)
        assert e.value.status == rb.RB_ENOENT
    finally:
        dep.destroy()


@pytest.mark.parametrize("name,n", [("multi_tenant", 400), ("ragged_seq", 120), ("large_mlp", 200)])
def test_serving_api_launch_windows(ctx, name, n):
    # rb_run_window: each launch window the clock dispatches (here up to 8
    # batches, several queues and models in one window) runs as one staged
    # copy and one launch chain per queue; every request's rows are
    # bit-identical to the replay's, which the oracle checks
    w = synth.workload(name)
    t, a = trace_and_arenas(name, n)
    *_, out_ref, out_off = run(ctx, name, n)
    check_outputs(name, t, a, out_ref, out_off, range(0, t.n, 3))
    dep = Deployment(w, ctx, device=True, window_batches=8, service_ns=service_table(w, base=10_000_000))
    sizes, queues_in_window = [], []
    try:
        def drain():
            while True:
                win = dep.sched.run_window()
                if win is None:
                    return
                sizes.append(len(win))
                queues_in_window.append(len({b["queue"] for b in win}))
        ids = []
        r = 0
        while r < t.n:
            tt = int(t.arrival_ns[r])
            while r < t.n and int(t.arrival_ns[r]) == tt:
                p = a.payload(r)
                ids.append(dep.sched.submit(dep.queue_for(t, r), int(t.n_rows[r]), p.dense, p.lens, p.ids,
                                            arrival_ns=tt))
                r += 1
            drain()
        for q, qc in zip(dep.queues, w.queues):
            if qc.timeout_ns is None:
                rb.check(rb.lib().rb_flush(q.h), "rb_flush")
        dep.sched.advance(int(t.arrival_ns[-1]) + 10 ** 12)
        drain()
        dep.sched.sync()
        for r in range(t.n):
            d_out = dep.models[int(t.servable[r])].d_out
            y = dep.sched.collect(ids[r], int(t.n_rows[r]), d_out)
            assert np.array_equal(y.ravel(), out_ref[out_off[r]:out_off[r + 1]]), r
    finally:
        dep.destroy()
    assert max(sizes) > 1
    if len(w.queues) > 1:
        assert max(queues_in_window) > 1
    print(f"{name}: {len(sizes)} windows, largest {max(sizes)} batches")


def test_destroy_old_version_while_its_batches_run(ctx):
    # availability-preserving swap right after an asynchronous replay, with no
    # sync: the old version is destroyed while its batches may still be
    # running. They hold references of their own, so its memory goes to the
    # deleter thread only after they finish; 2 GB of fresh allocations filled
    # with NaN right after the destroy must not reach any output, which must
    # equal an undisturbed replay's bit for bit. The new version then serves.
    name = "large_mlp"
    n = 1500
    w = synth.workload(name)
    t, a = trace_and_arenas(name, n)
    *_, out_ref, out_off = run(ctx, name, n, window=4)
    dep = Deployment(w, ctx, device=True, window_batches=4, service_ns=service_table(w))
    try:
        p_new = synth.next_version(synth.model_params(w, 0))
        new = dep.build_model(0, p_new)
        dt = dep.upload(t, a)
        dep.replay(dt)
        old = dep.swap(0, new)
        old.destroy()
        junk = [torch.full((64 << 20,), float("nan"), device="cuda") for _ in range(8)]
        dep.sched.sync()
        torch.cuda.synchronize()
        assert np.array_equal(dt.out.cpu().numpy(), out_ref)
        del junk
        dep.replay(dt)
        dep.sched.sync()
        out = dt.out.cpu().numpy()
        om_new = OracleModel(w.models[0], p_new)
        for r in range(0, n, 97):
            ref = om_new.forward(a.payload(r))
            y = out[out_off[r]:out_off[r + 1]].reshape(ref.shape)
            assert row_scaled_err(y, ref.astype(np.float64)) <= RTOL["bf16"], r
    finally:
        dep.destroy()


def _run_groups(ctx, name, n, groups, seq_pack, entry):
    """Every group of oracle-formed batches through one launch-group entry
    point, on torch's stream, into one output arena; returns it."""
    w = synth.workload(name)
    t, a = trace_and_arenas(name, n)
    dep = Deployment(w, ctx, device=True, seq_pack=seq_pack)
    try:
        dt = dep.upload(t, a)
        out = torch.zeros_like(dt.out)
        stream = rb.torch_stream_ptr()
        for grp in groups:
            kb, kr, slots, tokens = group_descriptors(w, t, a, dt.out_off, grp, seq_pack)
            kb_d = torch.from_numpy(kb.view(np.uint8).copy()).cuda()
            kr_d = torch.from_numpy(kr.view(np.uint8).copy()).cuda()
            lens_len = 0 if dt.lens is None else dt.lens.numel()
            ids_len = 0 if dt.ids is None else dt.ids.numel()
            dep.queues[grp[0].queue].run_group(stream, kb_d, len(kb), kr_d, len(kr), slots, tokens, dt.dense,
                                               dt.dense.numel(), dt.lens, lens_len, dt.ids, ids_len, out,
                                               out.numel(), entry=entry)
            torch.cuda.synchronize()
        dep.sched.sync()
        return out.cpu().numpy(), dt.out_off
    finally:
        dep.destroy()


def _oracle_groups(name, n, sizes):
    """Consecutive batches of each queue (as the oracle forms them), cut into
    groups of the given numbers of batches."""
    w = synth.workload(name)
    t, _ = trace_and_arenas(name, n)
    res = oracle_sim(w, t, service_table(w))
    groups = []
    for qi in range(len(w.queues)):
        mine = [b for b in res.batches if b.queue == qi]
        k = 0
        for sz in sizes:
            if k + sz <= len(mine):
                groups.append(mine[k:k + sz])
            k += sz
    return groups


@pytest.mark.parametrize("name,n,pack", [("small_mlp", 256, False), ("ranking", 600, False),
                                         ("large_mlp", 300, False), ("ragged_seq", 300, False),
                                         ("ragged_seq", 300, True)])
def test_run_group_matches_replay_and_oracle(ctx, name, n, pack):
    # rb_run_group on descriptors built outside the library: every request of
    # the groups gets the replay's rows bit for bit (same kernels, same row
    # independence), within tolerance of the oracle; requests in no group get
    # nothing
    groups = _oracle_groups(name, n, (3, 1, 2))
    assert groups
    *_, out_ref, out_off = run(ctx, name, n)
    out, _ = _run_groups(ctx, name, n, groups, pack, "rb_run_group")
    t, a = trace_and_arenas(name, n)
    covered = sorted(r for g in groups for b in g for r in b.reqs)
    for r in covered:
        assert np.array_equal(out[out_off[r]:out_off[r + 1]], out_ref[out_off[r]:out_off[r + 1]]), r
    mask = np.ones(out.size, bool)
    for r in covered:
        mask[out_off[r]:out_off[r + 1]] = False
    assert not out[mask].any()
    check_outputs(name, t, a, out, out_off, covered[::3])


def test_run_group_rejects_bad_descriptors(ctx):
    # descriptors whose rows, requests or output rows lie outside the extents
    # given: nothing is written out of bounds, the request gets no output, the
    # next rb_sync reports RB_ERANGE, and a good group still runs afterwards
    name = "small_mlp"
    w = synth.workload(name)
    t, a = trace_and_arenas(name, 64)
    grp = _oracle_groups(name, 64, (2,))[0]
    dep = Deployment(w, ctx, device=True)
    try:
        dt = dep.upload(t, a)
        stream = rb.torch_stream_ptr()
        kb0, kr0, slots, _ = group_descriptors(w, t, a, dt.out_off, grp)
        bads = []
        kb = kb0.copy(); kb[1]["row_base"] += 1; bads.append((kb, kr0))          # rows past the row map
        kb = kb0.copy(); kb[1]["n_req"] += 5; bads.append((kb, kr0))             # requests past the table
        kr = kr0.copy(); kr[0]["out_off"] = dt.out.numel(); bads.append((kb0, kr))  # output past the arena
        for kb, kr in bads:
            out = torch.zeros(dt.out.numel() + 64, dtype=torch.float32, device="cuda")
            kb_d = torch.from_numpy(kb.view(np.uint8).copy()).cuda()
            kr_d = torch.from_numpy(kr.view(np.uint8).copy()).cuda()
            dep.queues[0].run_group(stream, kb_d, len(kb), kr_d, len(kr), slots, 0, dt.dense, dt.dense.numel(),
                                    None, 0, None, 0, out, dt.out.numel())
            torch.cuda.synchronize()
            with pytest.raises(rb.RBError) as e:
                dep.sched.sync()
            assert e.value.status == rb.RB_ERANGE
            assert not out[dt.out.numel():].any()
        kb_d = torch.from_numpy(kb0.view(np.uint8).copy()).cuda()
        kr_d = torch.from_numpy(kr0.view(np.uint8).copy()).cuda()
        dep.queues[0].run_group(stream, kb_d, len(kb0), kr_d, len(kr0), slots, 0, dt.dense, dt.dense.numel(), None,
                                0, None, 0, dt.out, dt.out.numel())
        torch.cuda.synchronize()
        dep.sched.sync()
        check_outputs(name, t, a, dt.out.cpu().numpy(), dt.out_off, [r for b in grp for r in b.reqs])
    finally:
        dep.destroy()


def test_serving_api_ranking_and_seqpool(ctx):
    for name, n, pack in (("ranking", 120, False), ("ragged_seq", 60, False), ("ragged_seq", 60, True)):
        w = synth.workload(name)
        t, a = trace_and_arenas(name, n)
        dep = Deployment(w, ctx, device=True, seq_pack=pack)
        try:
            ids = []
            maxlen = dep.max_len(t)
            for r in range(t.n):
                p = a.payload(r)
                if name == "ragged_seq":
                    q = min((q for q in dep.queues if w.queues[dep.qindex[q.id]].bucket_len >= maxlen[r]),
                            key=lambda q: w.queues[dep.qindex[q.id]].bucket_len)
                else:
                    q = dep.queues[0]
                ids.append(dep.sched.submit(q, int(t.n_rows[r]), p.dense, p.lens, p.ids, 0))
            for q in dep.queues:
                rb.check(rb.lib().rb_flush(q.h), "rb_flush")
            while dep.sched.run_next() is not None:
                pass
            dep.sched.sync()
            for r in range(t.n):
                om = oracle_model(name, 0)
                ref = om.forward(a.payload(r))
                y = dep.sched.collect(ids[r], int(t.n_rows[r]), ref.shape[1])
                assert row_scaled_err(y, ref.astype(np.float64)) <= RTOL[w.models[0].dtype]
        finally:
            dep.destroy()


def test_device_bounds_errors_are_reported(ctx):
    # an id outside its table and bag lengths that disagree with the ids are
    # caught by the kernels' own bounds checks: nothing is read out of bounds
    name = "ranking"
    w = synth.workload(name)
    t, a = trace_and_arenas(name, 40)
    dep = Deployment(w, ctx, device=True)
    try:
        bad_ids = a.ids.copy()
        bad_ids[5] = 100_000_000
        a2 = synth.Arenas(a.dense, a.lens, bad_ids, a.dense_off, a.lens_off, a.ids_off)
        dt = dep.upload(t, a2)
        dep.replay(dt)
        with pytest.raises(rb.RBError) as e:
            dep.sched.sync()
        assert e.value.status == rb.RB_ERANGE
        bad_lens = a.lens.copy()
        bad_lens[3] += 1
        a3 = synth.Arenas(a.dense, bad_lens, a.ids, a.dense_off, a.lens_off, a.ids_off)
        dt = dep.upload(t, a3)
        dep.replay(dt)
        with pytest.raises(rb.RBError) as e:
            dep.sched.sync()
        assert e.value.status == rb.RB_ERANGE
        # the scheduler keeps serving afterwards
        dt = dep.upload(t, a)
        dep.replay(dt)
        dep.sched.sync()
    finally:
        dep.destroy()


def test_packed_tokens_bounds_errors_are_reported(ctx):
    # sequence lengths that disagree with a request's tokens: the routing
    # rejects the request, the packed rows of the others stay where the host
    # put them, and the scheduler keeps serving
    name = "ragged_seq"
    w = synth.workload(name)
    t, a = trace_and_arenas(name, 200)
    dep = Deployment(w, ctx, device=True, window_batches=8, seq_pack=True)
    try:
        for k in (3, 40):
            bad_lens = a.lens.copy()
            bad_lens[k] += 1 if k == 3 else 10_000
            a2 = synth.Arenas(a.dense, bad_lens, a.ids, a.dense_off, a.lens_off, a.ids_off)
            dt = dep.upload(t, a2)
            dep.replay(dt)
            with pytest.raises(rb.RBError) as e:
                dep.sched.sync()
            assert e.value.status == rb.RB_ERANGE
        dt = dep.upload(t, a)
        dep.replay(dt)
        dep.sched.sync()
        check_outputs(name, t, a, dt.out.cpu().numpy(), dt.out_off, range(t.n))
    finally:
        dep.destroy()


def test_version_transition_while_serving(ctx):
    # availability-preserving transition (the paper's Aspired Versions
    # Manager): a new version of a ranking servable is loaded on another
    # thread while the scheduler replays the trace, then replaces the old one
    import threading
    name = "multi_tenant"
    w = synth.workload(name)
    t, a = trace_and_arenas(name, 1500)
    S = 4  # a ranking model (26 tables of 100k rows)
    dep = Deployment(w, ctx, device=True, window_batches=16, service_ns=service_table(w), n_streams=4)
    try:
        dt = dep.upload(t, a)
        dep.replay(dt)
        dep.sched.sync()
        out1 = dt.out.cpu().numpy()
        p2 = synth.next_version(synth.model_params(w, S))
        loaded = {}
        th = threading.Thread(target=lambda: loaded.setdefault("m", dep.build_model(S, p2)))
        th.start()
        for _ in range(3):  # serving goes on while the new version loads
            dep.replay(dt)
            dep.sched.sync()
            assert np.array_equal(dt.out.cpu().numpy(), out1)
        th.join()
        old = dep.swap(S, loaded["m"])
        old.destroy()
        dep.replay(dt)
        dep.sched.sync()
        out2 = dt.out.cpu().numpy()
    finally:
        dep.destroy()
    mine = np.nonzero(t.servable == S)[0]
    others = np.nonzero(t.servable != S)[0]
    assert len(mine) > 10
    for r in others:
        o0, o1 = int(dt.out_off[r]), int(dt.out_off[r + 1])
        assert np.array_equal(out2[o0:o1], out1[o0:o1]), r
    om2 = OracleModel(w.models[S], p2)
    for r in mine[::3]:
        ref = om2.forward(a.payload(r)).astype(np.float64)
        y = out2[int(dt.out_off[r]):int(dt.out_off[r + 1])].reshape(ref.shape)
        assert row_scaled_err(y, ref) <= RTOL["bf16"], r
        assert not np.array_equal(y, out1[int(dt.out_off[r]):int(dt.out_off[r + 1])].reshape(ref.shape))


def test_resource_preserving_transition_serving_api(ctx):
    # resource-preserving policy: servable S's queue is held, its old version
    # destroyed before the new one is loaded; requests arriving meanwhile wait
    # while the other servables are served, then run on the new version
    name = "multi_tenant"
    w = synth.workload(name)
    t, a = trace_and_arenas(name, 400)
    S = 0  # an fp32 MLP tenant
    dep = Deployment(w, ctx, device=True)
    try:
        half = t.n // 2
        ids = {}

        def submit(rs):
            for r in rs:
                p = a.payload(r)
                q = dep.servables[int(t.servable[r])][0]
                ids[r] = dep.sched.submit(q, int(t.n_rows[r]), p.dense, p.lens, p.ids, int(t.arrival_ns[r]))
            for q in dep.queues:
                rb.check(rb.lib().rb_flush(q.h), "rb_flush")

        def drain():
            ran = []
            while (b := dep.sched.run_next()) is not None:
                ran.extend(b["reqs"])
            return ran

        submit(range(half))
        drain()
        q = dep.servables[S][0]
        q.set_model(None)
        dep.models[S].destroy()
        submit(range(half, t.n))
        ran = drain()
        held = [r for r in range(half, t.n) if int(t.servable[r]) == S]
        assert held and not set(ids[r] for r in held) & set(ran)
        p2 = synth.next_version(synth.model_params(w, S))
        dep.models[S] = dep.build_model(S, p2)
        q.set_model(dep.models[S])
        drain()
        dep.sched.sync()
        for r in range(t.n):
            s = int(t.servable[r])
            om = OracleModel(w.models[S], p2) if (s == S and r >= half) else oracle_model(name, s)
            ref = om.forward(a.payload(r)).astype(np.float64)
            y = dep.sched.collect(ids[r], int(t.n_rows[r]), ref.shape[1])
            assert row_scaled_err(y, ref) <= RTOL[w.models[s].dtype], (r, s)
    finally:
        dep.destroy()
