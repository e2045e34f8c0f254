"""The algorithmic work behind bench.py's roofline figures, counted again from
the batch log of a no-device replay: every dense layer's flops from the padded
batch sizes and the model's real dimensions, the weights once per launch group
(one queue's batches inside one launch window), and the split of the layers
between the kernels that run them (two GEMM layers and the fused last layer
with its head for the ranking MLP, the opt-in fused tail, the three layers of
the large MLP, the last of which writes the requests' outputs itself); and the
latency calibration's fit of the launch-window device model, tied to the
library's simulated clock."""
import numpy as np
import pytest

import bench
import synth
from paper_1712_06139_amd import rb
from paper_1712_06139_amd.deploy import Deployment

W = 64


@pytest.fixture(scope="module")
def ctx():
    return rb.Ctx(-1)


def _replay(ctx, name, n):
    w = synth.workload(name)
    t = synth.trace(w, n)
    a = synth.arenas(t)
    dep = Deployment(w, ctx, device=False, with_params=False, window_batches=W)
    try:
        logd = dep.replay_meta(t)
        qindex = dict(dep.qindex)
    finally:
        dep.destroy()
    return w, t, a, logd, qindex


def _padded(logd):
    nb = int(logd["n_batches"])
    return np.asarray(logd["b_padded"][:nb], np.int64), np.asarray(logd["b_queue"][:nb])


def _groups(logd):
    # (launch window, queue) pairs: consecutive windows of W dispatched batches
    P, q = _padded(logd)
    return len({(b // W, int(q[b])) for b in range(len(P))})


def test_ranking_layers_split_between_gemm_and_fused_head(ctx):
    w, t, a, logd, qindex = _replay(ctx, "ranking", 3000)
    P, _ = _padded(logd)
    m = w.models[0]
    dims = [(L.fan_in, L.fan_out) for L in m.layers]
    assert dims == [(1677, 1024), (1024, 512), (512, 256), (256, 1)]
    work = bench.algorithmic_work(w, t, a, logd, qindex, W)
    rows = int(P.sum())
    assert work["gemm_bf16"]["flops"] == 2 * rows * (1677 * 1024 + 1024 * 512)
    assert work["gemm_head"]["flops"] == 2 * rows * (512 * 256) + 2 * rows * 256
    assert "head" not in work and "mlp_tail" not in work
    g = _groups(logd)
    # inputs and outputs of every row plus the two layers' weights once per group
    assert work["gemm_bf16"]["bytes"] == 2 * (rows * (1677 + 1024 + 1024 + 512) + g * (1677 * 1024 + 1024 * 512))
    real = int(t.n_rows.sum())
    assert work["gemm_head"]["bytes"] == rows * 512 * 2 + g * (512 * 256 + 256) * 2 + real * 4 + rows * 32
    # the embedding bags: every id's 4-byte index and 128-byte table row, the
    # lengths and dense features of real rows, the bf16 output and row map of
    # every padded row
    n_ids = int(a.ids_off[-1])
    assert work["embbag"]["bytes"] == (rows * 32 + real * (26 * 4 + 13 * 4) + n_ids * (4 + 128)
                                       + rows * (26 * 64 + 13) * 2)


def test_ranking_fused_tail_accounting(ctx):
    w, t, a, logd, qindex = _replay(ctx, "ranking", 2000)
    P, _ = _padded(logd)
    rows = int(P.sum())
    work = bench.algorithmic_work(w, t, a, logd, qindex, W, fused=True)
    assert work["gemm_bf16"]["flops"] == 2 * rows * 1677 * 1024
    assert work["mlp_tail"]["flops"] == 2 * rows * (1024 * 512 + 512 * 256 + 256)
    assert "gemm_head" not in work


def test_large_mlp_weights_once_per_launch_group(ctx):
    w, t, a, logd, qindex = _replay(ctx, "large_mlp", 600)
    P, _ = _padded(logd)
    rows = int(P.sum())
    work = bench.algorithmic_work(w, t, a, logd, qindex, W)
    layers = [(4096, 8192), (8192, 8192), (8192, 4096)]
    assert work["gemm_bf16"]["flops"] == sum(2 * rows * k * n for k, n in layers)
    g = _groups(logd)
    real = int(t.n_rows.sum())
    # the last layer writes only the real rows' fp32 outputs, through the row
    # map, into the requests' output rows (no separate split)
    assert "split" not in work
    assert work["gemm_bf16"]["bytes"] == (2 * sum(rows * (k + n) + g * k * n for k, n in layers[:-1])
                                          + 2 * (rows * 8192 + g * 8192 * 4096) + real * 4096 * 4 + rows * 32)
    # real fp32 inputs read once, every padded row written in bf16, the row map
    assert work["assemble"]["bytes"] == real * 4096 * 4 + rows * 4096 * 2 + rows * 32


def test_chain_model_fit_recovers_the_device_model(ctx):
    # the three timings a device with chain time b, per-batch time S and tail
    # c would give are fitted back to (S, b, c); and the library's simulated
    # clock, given those values, completes a lone request exactly one lone
    # chain c1 = b + S + c after it closes
    b, S, c = 30_000, 5_000, 40_000
    nb, nw = 100, 2
    c1, T1, TW = b + S + c, b + S, nw * b + nb * S
    assert bench.chain_model_fit(c1, T1, TW, nb, nw) == (S, b, c)
    assert bench.chain_model_fit(c1, T1, nw * T1, nb, nw) == (1.0, T1 - 1.0, c)  # S clamped
    assert bench.chain_model_fit(T1 - 5, T1, TW, nb, nw)[2] == 0.0                   # tail clamped
    svc = [0] * 513
    svc[512] = S
    sched = rb.Sched(ctx, device=False, window_batches=W)
    m = rb.Model(ctx, "mlp", "f32", [(None, None, "none")], shapes=[(4, 4)])
    q = rb.Queue(sched, m, 512, (512,), None, 0, svc, b, c)
    try:
        log = sched.sim_run([[q]], np.array([0]), np.array([1_000]), np.array([512]))
        assert int(log["n_batches"]) == 1
        assert int(log["req_done_ns"][0]) - 1_000 == c1
    finally:
        q.destroy()
        sched.destroy()
        m.destroy()


def test_bench_refuses_more_than_one_gpu():
    # one GPU only: a request for several exits with a message before any
    # device work (no GPU is needed to check this)
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    for args, env in ((["--gpus", "2"], {}), ([], {"WORLD_SIZE": "4"})):
        r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), *args], capture_output=True, text=True,
                           timeout=120, env=dict(os.environ, **env))
        assert r.returncode != 0
        assert "one MI355X only" in r.stderr
        assert r.stdout.strip() == ""


@pytest.mark.parametrize("name,ns", [("multi_tenant", 2_000.0), ("multi_tenant", 200_000.0), ("small_mlp", 150_000.0)])
def test_cpu_latency_is_a_fifo_queue(name, ns):
    # the CPU oracle's latency model against Lindley's recursion for the same
    # single-server FIFO queue (waiting time W_{r+1} = max(0, W_r + S_r - A_{r+1})
    # with A the interarrival times): the same percentiles
    w = synth.workload(name)
    t = synth.trace(w, min(w.n_requests, 3000))
    out = bench.cpu_latency(w, t, ns, n_max=3000)
    n = out["requests"]
    S = t.n_rows[:n].astype(np.float64) * ns

    def lindley(arr):
        arr = np.asarray(arr[:n], np.float64)
        W = np.zeros(n)
        for r in range(1, n):
            W[r] = max(0.0, W[r - 1] + S[r - 1] - (arr[r] - arr[r - 1]))
        lat = W + S
        return (round(bench.nearest_rank(lat, 0.5) / 1e3, 1), round(bench.nearest_rank(lat, 0.99) / 1e3, 1))
    if "trace_arrivals" in out:
        got = out["trace_arrivals"]
        assert (got["p50_us"], got["p99_us"]) == lindley(t.arrival_ns)
        assert got["unstable"] == (w.rate_per_s * S.mean() * 1e-9 >= 1.0)
    else:
        for rho in (0.5, 0.9):
            got = out[f"rho{rho}"]
            arr = synth.trace(w, n, rate_per_s=rho * 1e9 / float(S.mean())).arrival_ns
            assert (got["p50_us"], got["p99_us"]) == lindley(arr)
