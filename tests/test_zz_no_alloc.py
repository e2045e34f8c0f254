"""The allocation-free launch-group entry point (rb_run_group_static) against
rb_run_group, through the C ABI: two calls in a row on one stream, the second
on a smaller group, must give bit-identical outputs (the same kernels on
work buffers carved from the per-GPU static array instead of allocated ones),
and a group too large for the array is refused with RB_ESIZE before anything
runs."""
import functools

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth
from oracle import batching as ob
from paper_1712_06139_amd import rb
from paper_1712_06139_amd.deploy import Deployment

from helpers import group_descriptors, oracle_queues, oracle_req_queue, service_table

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    return rb.Ctx(0)


@functools.lru_cache(maxsize=None)
def _trace(name, n):
    w = synth.workload(name)
    t = synth.trace(w, n)
    return w, t, synth.arenas(t)


def _batches(name, n, qi):
    w, t, _ = _trace(name, n)
    res = ob.simulate(oracle_queues(w), oracle_req_queue(w, t).tolist(), t.arrival_ns, t.n_rows, service_table(w))
    return [b for b in res.batches if b.queue == qi]


def _run(ctx, name, n, groups, entry, seq_pack=False):
    """Each group through `entry`, one after the other on torch's stream,
    into one fresh output arena per group; returns the arenas."""
    w, t, a = _trace(name, n)
    dep = Deployment(w, ctx, device=True, seq_pack=seq_pack)
    outs = []
    try:
        dt = dep.upload(t, a)
        stream = rb.torch_stream_ptr()
        keep = []
        for grp in groups:
            kb, kr, slots, tokens = group_descriptors(w, t, a, dt.out_off, grp, seq_pack)
            kb_d = torch.from_numpy(kb.view(np.uint8).copy()).cuda()
            kr_d = torch.from_numpy(kr.view(np.uint8).copy()).cuda()
            out = torch.full_like(dt.out, -7.0)
            keep += [kb_d, kr_d]
            dep.queues[grp[0].queue].run_group(stream, kb_d, len(kb), kr_d, len(kr), slots, tokens, dt.dense,
                                               dt.dense.numel(), dt.lens, 0 if dt.lens is None else dt.lens.numel(),
                                               dt.ids, 0 if dt.ids is None else dt.ids.numel(), out, out.numel(),
                                               entry=entry)
            outs.append(out)
        torch.cuda.synchronize()
        dep.sched.sync()
        return [o.cpu().numpy() for o in outs]
    finally:
        dep.destroy()


@pytest.mark.parametrize("name,n,qi,pack", [("small_mlp", 256, 0, False), ("ranking", 600, 0, False),
                                            ("large_mlp", 70, 0, False), ("ragged_seq", 300, 1, True),
                                            ("ragged_seq", 300, 0, False), ("multi_tenant", 1500, 4, False)])
def test_static_entry_point_matches_allocating_one(ctx, name, n, qi, pack):
    bs = _batches(name, n, qi)
    # two calls in a row, the second on a smaller group
    groups = [bs[:3], bs[3:4]] if len(bs) >= 4 else [bs[:2], bs[:1]]
    if name in ("large_mlp", "ragged_seq"):
        # one batch per call (one 1024-row batch of the large MLP, or one
        # 64-sequence batch, is about what the array holds): the largest
        # padded size, then the smallest
        by_p = sorted(bs, key=lambda b: b.P)
        groups = [by_p[-1:], by_p[:1]]
        assert groups[1][0].P < groups[0][0].P
    ref = _run(ctx, name, n, groups, "rb_run_group", pack)
    got = _run(ctx, name, n, groups, "rb_run_group_static", pack)
    for g, r, o in zip(groups, ref, got):
        assert np.array_equal(r, o)
        assert (r != -7.0).sum() > 0
    print(f"{name}: groups of {[len(g) for g in groups]} batches bit-identical")


def test_static_entry_point_refuses_groups_beyond_its_array(ctx):
    name, n = "large_mlp", 100
    w, t, a = _trace(name, n)
    bs = _batches(name, n, 0)
    dep = Deployment(w, ctx, device=True)
    try:
        dt = dep.upload(t, a)
        out = torch.full_like(dt.out, -7.0)
        kb, kr, slots, _ = group_descriptors(w, t, a, dt.out_off, bs[:2])
        kb_d = torch.from_numpy(kb.view(np.uint8).copy()).cuda()
        kr_d = torch.from_numpy(kr.view(np.uint8).copy()).cuda()
        with pytest.raises(rb.RBError) as e:
            dep.queues[0].run_group(rb.torch_stream_ptr(), kb_d, len(kb), kr_d, len(kr), slots, 0, dt.dense,
                                    dt.dense.numel(), None, 0, None, 0, out, out.numel(),
                                    entry="rb_run_group_static")
        assert e.value.status == rb.RB_ESIZE
        torch.cuda.synchronize()
        dep.sched.sync()
        assert (out.cpu().numpy() == -7.0).all()
    finally:
        dep.destroy()
