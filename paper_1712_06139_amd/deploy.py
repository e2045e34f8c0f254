"""Deploy a synthetic serving workload on the library: one model per
servable, one batching queue per servable (per length bucket for sequence
models), one scheduler; replay request traces through rb_sim_run.

Marshalling only: parameters and traces come from the seeded generators in
`synth`, payload arenas are uploaded as torch device tensors, and everything
the batching path computes happens inside librbatch.so.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

from . import rb


@dataclasses.dataclass
class DeviceTrace:
    """A trace's payload arenas in device memory plus the host metadata."""
    n: int
    servable: np.ndarray
    arrival_ns: np.ndarray
    n_rows: np.ndarray
    max_len: Optional[np.ndarray]
    dense: object
    dense_off: np.ndarray
    lens: object
    lens_off: np.ndarray
    ids: object
    ids_off: np.ndarray
    out: object
    out_off: np.ndarray
    examples: int


class Deployment:
    def __init__(self, w, ctx: rb.Ctx, device: bool = True, window_batches: int = 1, pad_value: float = 0.0,
                 profile: int = 0, service_ns: Optional[Sequence[Sequence[int]]] = None,
                 with_params: bool = True, models: Optional[List[rb.Model]] = None, n_streams: int = 1,
                 seq_pack: bool = False, window_ns: Optional[Sequence[int]] = None,
                 window_tail_ns: Optional[Sequence[int]] = None, clocked_windows: bool = False,
                 emb_dedup: bool = False, fused_tail: bool = False):
        import synth
        self.w = w
        self.ctx = ctx
        self.owns_models = models is None
        self.models: List[rb.Model] = [] if models is None else list(models)
        for si, m in enumerate(w.models if models is None else ()):
            if with_params:
                self.models.append(self.build_model(si, synth.model_params(w, si)))
            else:
                shapes = [(L.fan_out, L.fan_in) for L in m.layers]
                if m.kind == "ranking":
                    shapes.append((m.n_tables, 0))
                layers = [(None, None, L.act) for L in m.layers]
                self.models.append(rb.Model(ctx, m.kind, m.dtype, layers, n_dense=m.n_dense,
                                            head=None if m.head is None else
                                            (np.zeros((m.head.fan_out, m.head.fan_in), np.float32),
                                             np.zeros(m.head.fan_out, np.float32), m.head.act),
                                            shapes=shapes, table_rows=m.table_rows))
        self.sched = rb.Sched(ctx, device=device, window_batches=window_batches, pad_value=pad_value,
                              profile=profile, n_streams=n_streams, seq_pack=seq_pack,
                              clocked_windows=clocked_windows, emb_dedup=emb_dedup, fused_tail=fused_tail)
        self.queues: List[rb.Queue] = []
        for qi, q in enumerate(w.queues):
            svc = None if service_ns is None else service_ns[qi]
            self.queues.append(rb.Queue(self.sched, self.models[q.servable], q.max_batch_size, q.allowed,
                                        q.timeout_ns, q.bucket_len, svc,
                                        0 if window_ns is None else int(window_ns[qi]),
                                        0 if window_tail_ns is None else int(window_tail_ns[qi])))
        self.servables = [[self.queues[qi] for qi, q in enumerate(w.queues) if q.servable == s]
                          for s in range(len(w.models))]
        self.qindex = {q.id: i for i, q in enumerate(self.queues)}

    def build_model(self, si: int, p) -> rb.Model:
        """Servable si's model with parameters p (a synth.Params); safe to call
        on another thread while the scheduler serves (a new version)."""
        m = self.w.models[si]
        layers = [(W, b, L.act) for (W, b), L in zip(p.weights, m.layers)]
        head = None if m.head is None else (p.head[0], p.head[1], m.head.act)
        return rb.Model(self.ctx, m.kind, m.dtype, layers, tables=p.tables or None, n_dense=m.n_dense, head=head)

    def swap(self, si: int, new: rb.Model) -> rb.Model:
        """Availability-preserving version transition of servable si: its
        queues dispatch to `new` from now on; returns the old version, which
        the caller destroys (its memory is freed off the inference path)."""
        old = self.models[si]
        for q in self.servables[si]:
            q.set_model(new)
        self.models[si] = new
        return old

    def queue_for(self, t, r: int) -> rb.Queue:
        """The queue request r of trace t is submitted to: its servable's
        queue, or for bucketed sequence queues the smallest bucket that holds
        the request's longest sequence (the replay's rule)."""
        qs = self.servables[int(t.servable[r])]
        if len(qs) == 1 or t.seq_lens is None:
            return qs[0]
        L = int(t.seq_lens[t.seq_off[r]:t.seq_off[r + 1]].max())
        return min((q for q in qs if q.bucket_len >= L), key=lambda q: q.bucket_len)

    def destroy(self):
        for q in self.queues:
            q.destroy()
        self.sched.destroy()
        if self.owns_models:
            for m in self.models:
                m.destroy()

    # -- traces ------------------------------------------------------------

    def max_len(self, t) -> Optional[np.ndarray]:
        if t.seq_lens is None:
            return None
        return np.maximum.reduceat(t.seq_lens, t.seq_off[:-1]).astype(np.int32)

    def out_offsets(self, t) -> np.ndarray:
        d_out = np.array([m.d_out for m in self.models], dtype=np.int64)[t.servable]
        off = np.zeros(t.n + 1, dtype=np.int64)
        np.cumsum(t.n_rows.astype(np.int64) * d_out, out=off[1:])
        return off

    def upload(self, t, arenas, device="cuda") -> DeviceTrace:
        import torch
        dense = torch.from_numpy(arenas.dense).to(device) if arenas.dense.size else torch.zeros(4, device=device)
        lens = torch.from_numpy(arenas.lens).to(device) if arenas.lens.size else None
        ids = torch.from_numpy(arenas.ids).to(device) if arenas.ids.size else None
        out_off = self.out_offsets(t)
        out = torch.empty(max(int(out_off[-1]), 1), dtype=torch.float32, device=device)
        torch.cuda.synchronize()
        return DeviceTrace(t.n, t.servable, t.arrival_ns, t.n_rows, self.max_len(t), dense, arenas.dense_off,
                           lens, arenas.lens_off if lens is not None else None, ids,
                           arenas.ids_off if ids is not None else None, out, out_off, int(t.n_rows.sum()))

    def replay(self, dt: DeviceTrace) -> dict:
        """Replay a device-resident trace (asynchronous on the device)."""
        return self.sched.sim_run(self.servables, dt.servable, dt.arrival_ns, dt.n_rows, dt.max_len,
                                  dt.dense, dt.dense_off, dt.lens, dt.lens_off, dt.ids, dt.ids_off, dt.out,
                                  dt.out_off)

    def replay_meta(self, t) -> dict:
        """Replay a trace's metadata only (no-device scheduler)."""
        return self.sched.sim_run(self.servables, t.servable, t.arrival_ns, t.n_rows, self.max_len(t))

    def outputs(self, dt: DeviceTrace, r: int) -> np.ndarray:
        d_out = self.models[int(dt.servable[r])].d_out
        o0, o1 = int(dt.out_off[r]), int(dt.out_off[r + 1])
        return dt.out[o0:o1].cpu().numpy().reshape(-1, d_out)
