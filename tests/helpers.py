"""Shared test plumbing: oracle-side queue configs and request routing for a
workload, service-time tables, and batch-log comparison."""
import numpy as np

from oracle import batching as ob


def oracle_queues(w):
    return [ob.QueueCfg(q.max_batch_size, tuple(q.allowed), q.timeout_ns, q.bucket_len) for q in w.queues]


def oracle_req_queue(w, t):
    qs = oracle_queues(w)
    members = {s: [i for i, q in enumerate(w.queues) if q.servable == s] for s in range(len(w.models))}
    out = np.empty(t.n, dtype=np.int64)
    for r in range(t.n):
        mem = members[int(t.servable[r])]
        L = 0
        if t.seq_lens is not None:
            L = int(t.seq_lens[t.seq_off[r]:t.seq_off[r + 1]].max())
        out[r] = ob.pick_queue(qs, mem, L)
    return out


def service_table(w, base=20_000, per_row=100):
    return [[base + per_row * P for P in range(q.max_batch_size + 1)] for q in w.queues]


def oracle_sim(w, t, svc, window=1, window_ns=None, window_tail_ns=None):
    return ob.simulate(oracle_queues(w), oracle_req_queue(w, t).tolist(), t.arrival_ns, t.n_rows, svc, window,
                       window_ns, window_tail_ns)


def lib_batches(log, qindex):
    out = []
    for i in range(log["n_batches"]):
        b0, b1 = log["b_req_begin"][i], log["b_req_begin"][i + 1]
        out.append((qindex[int(log["b_queue"][i])], log["b_reqs"][b0:b1].tolist(), int(log["b_real"][i]),
                    int(log["b_padded"][i]), int(log["b_close_ns"][i]), int(log["b_dispatch_ns"][i]),
                    int(log["b_done_ns"][i])))
    return out


def oracle_batches(res):
    return [(b.queue, list(b.reqs), b.s, b.P, b.close_ns, b.dispatch_ns, b.done_ns) for b in res.batches]


def group_descriptors(w, t, a, out_off, batches, seq_pack=False):
    """A launch group's device descriptors (rb_k_batch / rb_k_req records as
    numpy structured arrays) for batches of one queue formed by the oracle:
    requests keep the trace's arena offsets and output offsets. Returns
    (kb, kr, slots, tokens)."""
    from paper_1712_06139_amd import rb
    q = w.queues[batches[0].queue]
    m = w.models[q.servable]
    kb = np.zeros(len(batches), dtype=rb.K_BATCH_DTYPE)
    n_req = sum(len(b.reqs) for b in batches)
    kr = np.zeros(n_req, dtype=rb.K_REQ_DTYPE)
    row, ri, tok = 0, 0, 0
    for bi, b in enumerate(batches):
        kb[bi] = (ri, len(b.reqs), row, b.P, b.s, q.bucket_len if m.kind == "seqpool" else 0)
        for r in b.reqs:
            lo = a.lens_off[r] if a.lens.size else 0
            io0, io1 = (a.ids_off[r], a.ids_off[r + 1]) if a.ids.size else (0, 0)
            kr[ri] = (a.dense_off[r], a.dense_off[r + 1], lo, io0, io1, out_off[r], t.n_rows[r], tok)
            if m.kind == "seqpool":
                tok += int(a.dense_off[r + 1] - a.dense_off[r]) // m.d_in
            ri += 1
        row += b.P
    return kb, kr, row, (tok if (m.kind == "seqpool" and seq_pack) else 0)
