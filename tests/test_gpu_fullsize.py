"""Full-size GPU parity, in the launch configuration bench.py times (window
of 64 dispatched batches): every workload's whole trace is replayed on the
GPU; the batch log must equal the oracle's bit for bit, and a seeded sample
of requests (the first and last, every request of the first and last batch,
one request of every distinct padded size, and random others) must match the
oracle's unbatched forward within tolerance."""
import functools

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth
from oracle.models import OracleModel
from paper_1712_06139_amd import rb
from paper_1712_06139_amd.deploy import Deployment

from helpers import lib_batches, oracle_batches, oracle_sim, service_table

pytestmark = pytest.mark.gpu

WINDOW = 64
RTOL = {"f32": 1e-5, "bf16": 2e-2}
N_RANDOM = {"ranking": 150, "large_mlp": 24, "multi_tenant": 150, "ragged_seq": 100}


@pytest.fixture(scope="module")
def ctx():
    return rb.Ctx(0)


@functools.lru_cache(maxsize=None)
def oracle_model(name, s):
    w = synth.workload(name)
    return OracleModel(w.models[s], synth.model_params(w, s))


def sample(log, n, rng, k):
    b0 = log["b_reqs"][log["b_req_begin"][0]:log["b_req_begin"][1]]
    nb = log["n_batches"]
    bl = log["b_reqs"][log["b_req_begin"][nb - 1]:log["b_req_begin"][nb]]
    pick = {0, n - 1, *b0.tolist(), *bl.tolist()}
    for P in np.unique(log["b_padded"]):
        i = int(np.nonzero(log["b_padded"] == P)[0][0])
        pick.add(int(log["b_reqs"][log["b_req_begin"][i]]))
    pick.update(rng.choice(n, size=k, replace=False).tolist())
    return sorted(pick)


@pytest.mark.parametrize("name", ["ranking", "large_mlp", "multi_tenant", "ragged_seq"])
def test_full_trace(ctx, name):
    w = synth.workload(name)
    t = synth.trace(w)
    a = synth.arenas(t)
    svc = service_table(w)
    dep = Deployment(w, ctx, device=True, window_batches=WINDOW, service_ns=svc)
    try:
        dt = dep.upload(t, a)
        log = dep.replay(dt)
        dep.sched.sync()
        ours = lib_batches(log, dep.qindex)
        out_off = dt.out_off
        reqs = sample(log, t.n, np.random.default_rng(2024), N_RANDOM[name])
        outs = {r: dt.out[int(out_off[r]):int(out_off[r + 1])].cpu().numpy() for r in reqs}
        del dt
    finally:
        dep.destroy()
    assert ours == oracle_batches(oracle_sim(w, t, svc, WINDOW))
    worst = 0.0
    for r in reqs:
        s = int(t.servable[r])
        ref = oracle_model(name, s).forward(a.payload(r)).astype(np.float64)
        y = outs[r].reshape(ref.shape).astype(np.float64)
        assert np.isfinite(y).all(), r
        e = float(np.max(np.abs(y - ref) / np.maximum(np.max(np.abs(ref), axis=1, keepdims=True), 1e-30)))
        worst = max(worst, e)
        assert e <= RTOL[w.models[s].dtype], (name, r, e)
    print(f"{name}: {t.n} requests, {len(ours)} batches, {len(reqs)} sampled, worst row-scaled error {worst:.3g}")


def test_full_ragged_seq_packed_tokens_bit_identical(ctx):
    # the whole ragged-sequence trace with the token-wise layers on packed
    # real tokens: the same batches, and every output bit-identical to the
    # padded path (whose sampled outputs test_full_trace checks against the
    # oracle)
    name = "ragged_seq"
    w = synth.workload(name)
    t = synth.trace(w)
    a = synth.arenas(t)
    svc = service_table(w)
    logs, outs = [], []
    for pack in (False, True):
        dep = Deployment(w, ctx, device=True, window_batches=WINDOW, service_ns=svc, seq_pack=pack)
        try:
            dt = dep.upload(t, a)
            log = dep.replay(dt)
            dep.sched.sync()
            logs.append(lib_batches(log, dep.qindex))
            outs.append(dt.out.cpu().numpy())
            del dt
        finally:
            dep.destroy()
    assert logs[0] == logs[1]
    assert np.isfinite(outs[1]).all()
    assert np.array_equal(outs[0], outs[1])
