"""Seeded synthetic serving workloads: request traces and model parameters.

This module only draws random numbers and lays them out. It holds none of the
batching method's arithmetic: no batch formation, no padding, no row routing,
no model evaluation and no rounding to bf16. The CPU oracle and the GPU path
both read what it produces, each doing its own arithmetic on it.

Five workloads stand in for the request streams a batching server sees
(paper section 2.2.1, "Inter-Request Batching": small requests for one or more
servables, merged by concatenating their input tensors):

  small_mlp     fp32 MLP 64->128(ReLU)->16; 256 requests of 1..8 rows;
                max batch 32, allowed sizes {8,16,32}; count-only batching.
  ranking       26 sum-pooled embedding bags (1..20 ids each, Zipf(1.1) over
                100k-row x 64 tables) + 13 dense features -> MLP
                1677->1024->512->256->1 (ReLU, sigmoid out), bf16 weights;
                100k requests of 1..64 rows; max 512, allowed {64,...,512}.
  large_mlp     bf16 MLP 4096->8192->8192->4096 (ReLU hidden, linear out);
                20k requests of 1..32 rows; max 1024, allowed {128,...,1024}.
  multi_tenant  8 servables: 4 fp32 MLPs 256->1024->1024->32 and 4 ranking
                models with distinct seeds; Poisson arrivals at 50k req/s,
                servable chosen Zipf(1.0); 1..16 rows; max 256, no padding,
                2 ms batch timeout.
  ragged_seq    requests of 1..4 sequences of 1..512 tokens (log-uniform),
                256-dim tokens; per-token MLP 256->512(ReLU)->256, masked
                mean-pool, 256->2 softmax; one queue per length bucket
                {64,128,256,512}, max 64 sequences per batch.

Seeds: every stream is numpy PCG64 on SeedSequence([0x5EED, workload id,
stream id, ...]). Request payloads are drawn per chunk of CHUNK requests, so a
prefix of a trace equals the same prefix of the full trace, and any single
request can be regenerated without drawing the whole trace.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

SEED_ROOT = 0x5EED
CHUNK = 256  # requests per payload chunk

# stream ids
_S_ROWS, _S_ARRIVAL, _S_SERVABLE, _S_PAYLOAD, _S_SEQLEN = 1, 2, 3, 4, 5
_S_WEIGHT, _S_TABLE, _S_PERM = 100, 200, 300


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, *key])))


@dataclasses.dataclass(frozen=True)
class Layer:
    fan_in: int
    fan_out: int
    act: str  # "relu" | "none" | "sigmoid"


@dataclasses.dataclass(frozen=True)
class Model:
    """A served model. kind: "mlp" (dense rows), "ranking" (embedding bags +
    dense features -> MLP) or "seqpool" (per-token MLP, masked mean-pool,
    linear + softmax head)."""
    kind: str
    dtype: str                 # "f32" or "bf16" (bf16 storage, fp32 accumulation)
    layers: Tuple[Layer, ...]  # MLP after the embedding concat / per-token MLP
    seed_id: int
    init: str = "xavier"       # "xavier" or "normal_fanin"
    n_tables: int = 0
    table_rows: int = 0
    emb_dim: int = 0
    n_dense: int = 0
    bag_len: Tuple[int, int] = (0, 0)   # inclusive range of ids per bag
    zipf_s: float = 0.0
    head: Optional[Layer] = None        # seqpool head (softmax)

    @property
    def d_in(self) -> int:
        """Floats per request row in the dense payload."""
        if self.kind == "ranking":
            return self.n_dense
        return self.layers[0].fan_in

    @property
    def d_out(self) -> int:
        """Floats per request row in the output."""
        if self.kind == "seqpool":
            return self.head.fan_out
        return self.layers[-1].fan_out


@dataclasses.dataclass(frozen=True)
class Queue:
    """One batching queue: a servable's queue (or one length bucket of it)."""
    servable: int
    max_batch_size: int
    allowed: Tuple[int, ...]       # allowed batch sizes; () = run at the real size
    timeout_ns: Optional[int]      # None = batches close by count only
    bucket_len: int = 0            # > 0: queue takes sequences up to this length


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int
    models: Tuple[Model, ...]      # one per servable
    queues: Tuple[Queue, ...]
    n_requests: int
    rows: Tuple[int, int]          # inclusive range of rows (sequences) per request
    rate_per_s: float              # default Poisson arrival rate
    servable_zipf_s: float = 0.0   # > 0: servable chosen Zipf(s) over models
    seq_len_max: int = 0           # ragged_seq: max tokens per sequence


def _ranking(seed_id: int) -> Model:
    return Model(kind="ranking", dtype="bf16", seed_id=seed_id,
                 layers=(Layer(26 * 64 + 13, 1024, "relu"), Layer(1024, 512, "relu"),
                         Layer(512, 256, "relu"), Layer(256, 1, "sigmoid")),
                 n_tables=26, table_rows=100_000, emb_dim=64, n_dense=13,
                 bag_len=(1, 20), zipf_s=1.1)


def _tenant_mlp(seed_id: int) -> Model:
    return Model(kind="mlp", dtype="f32", seed_id=seed_id,
                 layers=(Layer(256, 1024, "relu"), Layer(1024, 1024, "relu"), Layer(1024, 32, "none")))


WORKLOADS: Dict[str, Workload] = {}


def _register(w: Workload) -> None:
    WORKLOADS[w.name] = w


_register(Workload(
    name="small_mlp", wid=1,
    models=(Model(kind="mlp", dtype="f32", seed_id=0,
                  layers=(Layer(64, 128, "relu"), Layer(128, 16, "none"))),),
    queues=(Queue(0, 32, (8, 16, 32), None),),
    n_requests=256, rows=(1, 8), rate_per_s=100_000.0))

_register(Workload(
    name="ranking", wid=2,
    models=(_ranking(0),),
    queues=(Queue(0, 512, (64, 128, 256, 512), None),),
    n_requests=100_000, rows=(1, 64), rate_per_s=100_000.0))

_register(Workload(
    name="large_mlp", wid=3,
    models=(Model(kind="mlp", dtype="bf16", seed_id=0, init="normal_fanin",
                  layers=(Layer(4096, 8192, "relu"), Layer(8192, 8192, "relu"),
                          Layer(8192, 4096, "none"))),),
    queues=(Queue(0, 1024, (128, 256, 512, 1024), None),),
    n_requests=20_000, rows=(1, 32), rate_per_s=20_000.0))

_register(Workload(
    name="multi_tenant", wid=4,
    models=tuple([_tenant_mlp(i) for i in range(4)] + [_ranking(4 + i) for i in range(4)]),
    queues=tuple(Queue(m, 256, (), 2_000_000) for m in range(8)),
    n_requests=50_000, rows=(1, 16), rate_per_s=50_000.0, servable_zipf_s=1.0))

_register(Workload(
    name="ragged_seq", wid=5,
    models=(Model(kind="seqpool", dtype="f32", seed_id=0,
                  layers=(Layer(256, 512, "relu"), Layer(512, 256, "none")),
                  head=Layer(256, 2, "softmax")),),
    queues=tuple(Queue(0, 64, (), None, bucket_len=b) for b in (64, 128, 256, 512)),
    n_requests=50_000, rows=(1, 4), rate_per_s=50_000.0, seq_len_max=512))


def workload(name: str) -> Workload:
    return WORKLOADS[name]


# ---------------------------------------------------------------------------
# model parameters
# ---------------------------------------------------------------------------

def _layer_params(w: Workload, m: Model, li: int, layer: Layer) -> Tuple[np.ndarray, np.ndarray]:
    rng = _rng(w.wid, _S_WEIGHT + m.seed_id, li)
    if m.init == "normal_fanin":
        W = rng.standard_normal((layer.fan_out, layer.fan_in), dtype=np.float32)
        W *= np.float32(1.0 / math.sqrt(layer.fan_in))
    else:
        a = math.sqrt(6.0 / (layer.fan_in + layer.fan_out))
        W = rng.uniform(-a, a, size=(layer.fan_out, layer.fan_in)).astype(np.float32)
    bb = 1.0 / math.sqrt(layer.fan_in)
    b = rng.uniform(-bb, bb, size=layer.fan_out).astype(np.float32)
    return W, b


@dataclasses.dataclass
class Params:
    """fp32 draws of a model's parameters. W is [fan_out, fan_in] row-major."""
    weights: List[Tuple[np.ndarray, np.ndarray]]
    tables: List[np.ndarray]              # ranking: n_tables x [table_rows, emb_dim]
    head: Optional[Tuple[np.ndarray, np.ndarray]] = None


_param_cache: Dict[Tuple[str, int], Params] = {}


def next_version(p: Params) -> Params:
    """Parameters of a new version of a servable: weights halved, tables
    doubled (power-of-two scalings, so bf16 storage stays exact), biases
    shifted by 0.25 so that every output changes."""
    return Params([(W * np.float32(0.5), b + np.float32(0.25)) for W, b in p.weights],
                  [T * np.float32(2.0) for T in p.tables],
                  None if p.head is None else (p.head[0] * np.float32(0.5), p.head[1]))


def model_params(w: Workload, servable: int, cache: bool = True) -> Params:
    key = (w.name, servable)
    if cache and key in _param_cache:
        return _param_cache[key]
    m = w.models[servable]
    weights = [_layer_params(w, m, li, L) for li, L in enumerate(m.layers)]
    tables: List[np.ndarray] = []
    for t in range(m.n_tables):
        rng = _rng(w.wid, _S_TABLE + m.seed_id, t)
        T = rng.standard_normal((m.table_rows, m.emb_dim), dtype=np.float32)
        T *= np.float32(1.0 / 8.0)
        tables.append(T)
    head = _layer_params(w, m, len(m.layers), m.head) if m.head is not None else None
    p = Params(weights, tables, head)
    if cache:
        _param_cache[key] = p
    return p


# ---------------------------------------------------------------------------
# Zipf sampling (bounded, ranks 1..n, P(k) proportional to k^-s)
# ---------------------------------------------------------------------------

class _Alias:
    """Walker/Vose alias table: exact sampling from a finite distribution."""

    def __init__(self, p: np.ndarray):
        n = len(p)
        q = p / p.sum() * n
        prob = np.ones(n)
        alias = np.arange(n, dtype=np.int64)
        small = [i for i in range(n) if q[i] < 1.0]
        large = [i for i in range(n) if q[i] >= 1.0]
        while small and large:
            s = small.pop()
            g = large.pop()
            prob[s] = q[s]
            alias[s] = g
            q[g] = q[g] + q[s] - 1.0
            (small if q[g] < 1.0 else large).append(g)
        self.n = n
        self.prob = prob
        self.alias = alias.astype(np.int32)

    def sample(self, rng: np.random.Generator, size: int) -> np.ndarray:
        """0-based indices."""
        idx = rng.integers(0, self.n, size=size, dtype=np.int32)
        u = rng.random(size)
        return np.where(u < np.take(self.prob, idx), idx, np.take(self.alias, idx))


_alias_cache: Dict[Tuple[int, float], _Alias] = {}


def _zipf_alias(n: int, s: float) -> _Alias:
    key = (n, s)
    if key not in _alias_cache:
        k = np.arange(1, n + 1, dtype=np.float64)
        _alias_cache[key] = _Alias(k ** (-s))
    return _alias_cache[key]


_perm_cache: Dict[Tuple[int, int], np.ndarray] = {}


def _rank_to_row(w: Workload, m: Model) -> np.ndarray:
    """[n_tables, table_rows] int32: a seeded permutation per table mapping
    Zipf rank-1 to a table row, so hot rows are scattered over the table."""
    key = (w.wid, m.seed_id)
    if key not in _perm_cache:
        perms = np.empty((m.n_tables, m.table_rows), dtype=np.int32)
        for t in range(m.n_tables):
            perms[t] = _rng(w.wid, _S_PERM + m.seed_id, t).permutation(m.table_rows).astype(np.int32)
        _perm_cache[key] = perms
    return _perm_cache[key]


# ---------------------------------------------------------------------------
# trace metadata
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Trace:
    """Per-request metadata of a trace (request r in submission order).

    servable[r]  which servable the request calls
    arrival_ns[r] non-decreasing int64 arrival times
    n_rows[r]    rows of the request (examples; sequences for seqpool)
    seq_lens     seqpool: tokens per sequence, flat; seq_off[r] indexes it
    """
    workload: Workload
    servable: np.ndarray
    arrival_ns: np.ndarray
    n_rows: np.ndarray
    seq_lens: Optional[np.ndarray] = None
    seq_off: Optional[np.ndarray] = None

    @property
    def n(self) -> int:
        return int(self.n_rows.shape[0])


def poisson_arrivals(w: Workload, n: int, rate_per_s: float) -> np.ndarray:
    """Poisson process: exponential gaps, cumulative times floored to int64 ns."""
    gaps = _rng(w.wid, _S_ARRIVAL).exponential(1.0 / rate_per_s, size=n)
    return np.floor(np.cumsum(gaps) * 1e9).astype(np.int64)


def trace(w: Workload, n_requests: Optional[int] = None, rate_per_s: Optional[float] = None) -> Trace:
    """The first n_requests requests (default: all) of the workload's trace."""
    N = w.n_requests
    n = N if n_requests is None else int(n_requests)
    if n > N:
        raise ValueError(f"{w.name} has {N} requests")
    n_rows = _rng(w.wid, _S_ROWS).integers(w.rows[0], w.rows[1] + 1, size=N).astype(np.int32)[:n]
    arrival = poisson_arrivals(w, N, rate_per_s or w.rate_per_s)[:n]
    if w.servable_zipf_s > 0:
        k = len(w.models)
        servable = _zipf_alias(k, w.servable_zipf_s).sample(_rng(w.wid, _S_SERVABLE), N)[:n].astype(np.int32)
    else:
        servable = np.zeros(n, dtype=np.int32)
    t = Trace(w, servable, arrival, n_rows)
    if w.seq_len_max:
        # length L = clip(floor(exp(u * ln(Lmax + 1))), 1, Lmax), u ~ U[0,1)
        total = int(_rng(w.wid, _S_ROWS).integers(w.rows[0], w.rows[1] + 1, size=N).astype(np.int64).sum())
        u = _rng(w.wid, _S_SEQLEN).random(total)
        L = np.clip(np.floor(np.exp(u * math.log(w.seq_len_max + 1))), 1, w.seq_len_max).astype(np.int32)
        off = np.zeros(n + 1, dtype=np.int64)
        np.cumsum(n_rows, out=off[1:])
        t.seq_lens = L[: off[-1]]
        t.seq_off = off
    return t


# ---------------------------------------------------------------------------
# payloads
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Payload:
    """One request's input tensors (row-major).

    mlp:      dense [n, d_in] f32
    ranking:  dense [n, n_dense] f32, lens [n, n_tables] i32 (ids per bag),
              ids [sum(lens)] i32 table rows, example-major then table-minor
    seqpool:  dense [sum(L), d_in] f32 tokens, sequence after sequence;
              lens [n] i32 = tokens per sequence
    """
    dense: np.ndarray
    lens: Optional[np.ndarray] = None
    ids: Optional[np.ndarray] = None


@dataclasses.dataclass
class _Chunk:
    """Payloads of CHUNK consecutive requests, concatenated in request order."""
    dense: np.ndarray
    lens: np.ndarray
    ids: np.ndarray
    n_dense: np.ndarray   # per request element counts
    n_lens: np.ndarray
    n_ids: np.ndarray


def _draw_chunk(w: Workload, t: Trace, lo: int, hi: int, rng: np.random.Generator) -> _Chunk:
    """Draw the payloads of requests [lo, hi): servable after servable (in
    servable order), each tensor for all of that servable's requests at once,
    then laid out in request order."""
    n_req = hi - lo
    srv = t.servable[lo:hi]
    rows = t.n_rows[lo:hi].astype(np.int64)
    parts = {}
    for s in np.unique(srv):
        m = w.models[int(s)]
        sel = np.nonzero(srv == s)[0]
        nr = rows[sel]
        if m.kind == "mlp":
            d = rng.standard_normal((int(nr.sum()), m.d_in), dtype=np.float32)
            parts[int(s)] = (sel, d.reshape(-1), nr * m.d_in, None, np.zeros_like(nr), None, np.zeros_like(nr))
        elif m.kind == "seqpool":
            L = np.concatenate([t.seq_lens[t.seq_off[lo + i]:t.seq_off[lo + i + 1]] for i in sel])
            tok_per_req = np.add.reduceat(L.astype(np.int64), np.concatenate([[0], np.cumsum(nr)[:-1]]))
            d = rng.standard_normal((int(L.sum()), m.d_in), dtype=np.float32)
            parts[int(s)] = (sel, d.reshape(-1), tok_per_req * m.d_in, L.astype(np.int32), nr, None,
                             np.zeros_like(nr))
        else:
            tot_rows = int(nr.sum())
            dense = rng.standard_normal((tot_rows, m.n_dense), dtype=np.float32)
            lens = rng.integers(m.bag_len[0], m.bag_len[1] + 1, size=(tot_rows, m.n_tables)).astype(np.int32)
            ranks0 = _zipf_alias(m.table_rows, m.zipf_s).sample(rng, int(lens.sum()))
            table_of = np.repeat(np.tile(np.arange(m.n_tables, dtype=np.int64), tot_rows), lens.ravel())
            ids = np.take(_rank_to_row(w, m).ravel(), table_of * m.table_rows + ranks0)
            row_off = np.concatenate([[0], np.cumsum(nr)[:-1]])
            ids_per_req = np.add.reduceat(lens.sum(axis=1, dtype=np.int64), row_off) if tot_rows else nr * 0
            parts[int(s)] = (sel, dense.reshape(-1), nr * m.n_dense, lens.reshape(-1), nr * m.n_tables,
                             ids.astype(np.int32), ids_per_req)
    n_dense = np.zeros(n_req, np.int64)
    n_lens = np.zeros(n_req, np.int64)
    n_ids = np.zeros(n_req, np.int64)
    for sel, _, nd, _, nl, _, ni in parts.values():
        n_dense[sel], n_lens[sel], n_ids[sel] = nd, nl, ni
    if len(parts) == 1:
        (_, d, _, ln, _, ii, _), = parts.values()
        return _Chunk(d, ln if ln is not None else np.zeros(0, np.int32),
                      ii if ii is not None else np.zeros(0, np.int32), n_dense, n_lens, n_ids)
    # several servables: scatter each servable's slices back into request order
    def gather(idx_data, idx_cnt, counts, dtype):
        out = np.empty(int(counts.sum()), dtype=dtype)
        off = np.concatenate([[0], np.cumsum(counts)])
        for sel, *rest in parts.values():
            data, cnt = rest[idx_data - 1], rest[idx_cnt - 1]
            if data is None:
                continue
            src = np.concatenate([[0], np.cumsum(cnt)])
            for j, r in enumerate(sel):
                out[off[r]:off[r + 1]] = data[src[j]:src[j + 1]]
        return out
    return _Chunk(gather(1, 2, n_dense, np.float32), gather(3, 4, n_lens, np.int32),
                  gather(5, 6, n_ids, np.int32), n_dense, n_lens, n_ids)


_full_cache: Dict[str, Trace] = {}


def _full_trace(w: Workload) -> Trace:
    if w.name not in _full_cache:
        _full_cache[w.name] = trace(w)
    return _full_cache[w.name]


def _chunk(w: Workload, c: int) -> _Chunk:
    # a chunk is always drawn in full from the full trace's metadata, so a
    # prefix trace sees exactly the payloads of the full one
    full = _full_trace(w)
    lo, hi = c * CHUNK, min((c + 1) * CHUNK, w.n_requests)
    return _draw_chunk(w, full, lo, hi, _rng(w.wid, _S_PAYLOAD, c))


def _slice(ch: _Chunk, i: int, w: Workload, t: Trace, r: int) -> Payload:
    d0, l0, i0 = (int(x[:i].sum()) for x in (ch.n_dense, ch.n_lens, ch.n_ids))
    m = w.models[int(t.servable[r])]
    dense = ch.dense[d0:d0 + ch.n_dense[i]]
    lens = ch.lens[l0:l0 + ch.n_lens[i]]
    ids = ch.ids[i0:i0 + ch.n_ids[i]]
    if m.kind == "mlp":
        return Payload(dense.reshape(-1, m.d_in))
    if m.kind == "seqpool":
        return Payload(dense.reshape(-1, m.d_in), lens=lens)
    return Payload(dense.reshape(-1, m.n_dense), lens.reshape(-1, m.n_tables), ids)


def request_payload(t: Trace, r: int) -> Payload:
    w = t.workload
    return _slice(_chunk(w, r // CHUNK), r % CHUNK, w, _full_trace(w), r)


@dataclasses.dataclass
class Arenas:
    """All payloads of a trace, concatenated in request order.

    dense (f32), lens (i32), ids (i32) are flat; *_off[r] are element offsets
    of request r's first element (length n+1; the last entry is the total).
    """
    dense: np.ndarray
    lens: np.ndarray
    ids: np.ndarray
    dense_off: np.ndarray
    lens_off: np.ndarray
    ids_off: np.ndarray

    def payload(self, r: int) -> Payload:
        d = self.dense[self.dense_off[r]:self.dense_off[r + 1]]
        ln = self.lens[self.lens_off[r]:self.lens_off[r + 1]]
        ids = self.ids[self.ids_off[r]:self.ids_off[r + 1]]
        return Payload(d, ln if ln.size else None, ids if ids.size else None)


def arenas(t: Trace, threads: Optional[int] = None) -> Arenas:
    """Draw every request's payload and concatenate them (threads over chunks)."""
    w = t.workload
    n_chunks = (t.n + CHUNK - 1) // CHUNK
    threads = threads or min(16, len(os.sched_getaffinity(0)))
    _full_trace(w)
    with ThreadPoolExecutor(max_workers=threads) as ex:
        chunks = list(ex.map(lambda c: _chunk(w, c), range(n_chunks)))
    last = t.n - (n_chunks - 1) * CHUNK if n_chunks else 0

    def cat(field, counts_field):
        parts = []
        for i, ch in enumerate(chunks):
            a = getattr(ch, field)
            if i == n_chunks - 1:
                a = a[:int(getattr(ch, counts_field)[:last].sum())]
            parts.append(a)
        return np.concatenate(parts) if parts else np.zeros(0)

    def offs(counts_field):
        cnt = np.concatenate([getattr(ch, counts_field) for ch in chunks])[: t.n] if chunks else np.zeros(0, np.int64)
        o = np.zeros(t.n + 1, dtype=np.int64)
        np.cumsum(cnt, out=o[1:])
        return o

    return Arenas(cat("dense", "n_dense").astype(np.float32, copy=False), cat("lens", "n_lens").astype(np.int32, copy=False),
                  cat("ids", "n_ids").astype(np.int32, copy=False), offs("n_dense"), offs("n_lens"), offs("n_ids"))
