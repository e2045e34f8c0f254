"""Oracle forward passes of the served models, one request at a time.

Test infrastructure only: nothing on the product path imports this module.

The paper's batching layer treats a servable as a black box whose Run() is
called on a merged request (section 2.1, servables as opaque objects;
section 2.2.1, the batching Session wrapper forwards the concatenated inputs
to the wrapped Run() and hands each caller its part). A caller must get what
an unbatched Run() on its own request would have returned, so the oracle's
reference output for request r is the model applied to r's rows alone:
forward(payload_r). Three model kinds are served:

  mlp      rows of d_in floats -> dense layers
  ranking  per row: 26 sum-pooled embedding bags ++ 13 dense floats -> MLP
  seqpool  per sequence: per-token MLP, mean over the sequence's tokens,
           linear head, softmax

forward_batch() runs the same arithmetic on a concatenated, padded batch; it
exists so tests can show that batching (concat, pad, run once, split) gives
every caller exactly its unbatched result.
"""
from __future__ import annotations

from typing import List, Optional, Tuple

import numpy as np

from . import numerics as nx


class OracleModel:
    """A model with its parameters in storage precision (fp64 arrays holding
    fp32- or bf16-representable values)."""

    def __init__(self, model, params):
        self.model = model
        self.kind = model.kind
        self.dtype = model.dtype
        store = nx.round_bf16 if model.dtype == "bf16" else nx.round_f32
        # weights in storage precision, biases fp32
        self.layers: List[Tuple[np.ndarray, np.ndarray, str]] = [
            (store(W).astype(np.float32), np.asarray(b, np.float32), L.act)
            for (W, b), L in zip(params.weights, model.layers)]
        self.tables = [store(T).astype(np.float32) for T in params.tables]
        self.head = None
        if params.head is not None:
            W, b = params.head
            self.head = (nx.round_f32(W).astype(np.float32), np.asarray(b, np.float32), model.head.act)

    # -- building blocks -------------------------------------------------

    def _round_in(self, x: np.ndarray) -> np.ndarray:
        return nx.round_bf16(x) if self.dtype == "bf16" else nx.round_f32(x)

    def mlp(self, h: np.ndarray) -> np.ndarray:
        """Dense layers on rows of h (already in the model's input precision).

        fp32 models round every layer output to fp32. bf16 models round every
        hidden output to bf16 (it is the next layer's input) and the last
        layer's output to fp32; the activation comes before the rounding.
        """
        n = len(self.layers)
        for i, (W, b, act) in enumerate(self.layers):
            z = nx.dense(h, W, b, act)
            if self.dtype == "bf16" and i < n - 1:
                h = nx.round_bf16(z)
            else:
                h = nx.round_f32(z)
        return h

    def ranking_input(self, dense: np.ndarray, lens: np.ndarray, ids: np.ndarray) -> np.ndarray:
        """Rows of the first MLP layer's input for ranking rows.

        Row e is [pool_0 | pool_1 | ... | pool_25 | dense_e], where pool_f is
        the sum of table f's rows over bag (e, f), rounded to bf16, and the 13
        dense floats are rounded to bf16. Bags are stored row-major: the ids of
        row e's bag f follow those of bag f-1 (and row e-1's last bag).
        """
        m = self.model
        n = dense.shape[0]
        lens = np.asarray(lens, np.int64).reshape(n, m.n_tables)
        ids = np.asarray(ids, np.int64)
        # offset of each bag's first id, bags in row-major order
        bag_start = np.zeros(n * m.n_tables, dtype=np.int64)
        np.cumsum(lens.ravel()[:-1], out=bag_start[1:])
        bag_start = bag_start.reshape(n, m.n_tables)
        X = np.empty((n, m.n_tables * m.emb_dim + m.n_dense), dtype=np.float64)
        for f in range(m.n_tables):
            # ids of table f's bags, bag after bag
            seg = [ids[bag_start[e, f]: bag_start[e, f] + lens[e, f]] for e in range(n)]
            fid = np.concatenate(seg) if seg else np.zeros(0, np.int64)
            pooled = nx.embedding_bag_sums(self.tables[f], fid, lens[:, f])
            X[:, f * m.emb_dim:(f + 1) * m.emb_dim] = nx.round_bf16(pooled)
        X[:, m.n_tables * m.emb_dim:] = nx.round_bf16(dense)
        return X

    def seq_head(self, pooled: np.ndarray) -> np.ndarray:
        W, b, act = self.head
        logits = nx.round_f32(nx.dense(pooled, W, b, "none"))
        return nx.round_f32(nx.ACTS[act](logits))

    # -- per-request (unbatched) definition --------------------------------

    def forward(self, payload) -> np.ndarray:
        """Output rows [n, d_out] (float32) of one request run on its own."""
        m = self.model
        if self.kind == "mlp":
            return self.mlp(self._round_in(np.asarray(payload.dense).reshape(-1, m.d_in))).astype(np.float32)
        if self.kind == "ranking":
            X = self.ranking_input(np.asarray(payload.dense).reshape(-1, m.n_dense), payload.lens, payload.ids)
            return self.mlp(X).astype(np.float32)
        # seqpool: each sequence on its own, over its own tokens only
        lens = np.asarray(payload.lens, np.int64)
        toks = np.asarray(payload.dense).reshape(-1, self.model.d_in)
        out = []
        t0 = 0
        for L in lens:
            h = self.mlp(nx.round_f32(toks[t0:t0 + L]))
            t0 += L
            pooled = nx.round_f32(np.sum(h, axis=0) / L)
            out.append(self.seq_head(pooled[None, :])[0])
        return np.asarray(out, np.float32).reshape(len(lens), -1)

    # -- on a merged batch -------------------------------------------------

    def forward_batch(self, batch) -> np.ndarray:
        """Output rows [P, d_out] for an assembled, padded batch (see
        batching.assemble). Pad rows are computed like any other row."""
        if self.kind == "mlp":
            return self.mlp(self._round_in(batch.dense)).astype(np.float32)
        if self.kind == "ranking":
            X = self.ranking_input(batch.dense, batch.lens, batch.ids)
            return self.mlp(X).astype(np.float32)
        # seqpool: tokens [P, T, d]; masked mean over t < L, chosen by
        # selection so pad tokens (even NaN ones) never enter the sum
        P, T, d = batch.tokens.shape
        h = self.mlp(nx.round_f32(batch.tokens.reshape(P * T, d))).reshape(P, T, -1)
        L = np.asarray(batch.seq_len, np.int64)
        mask = np.arange(T)[None, :, None] < L[:, None, None]
        s = np.sum(np.where(mask, h, 0.0), axis=1)
        pooled = nx.round_f32(s / np.maximum(L, 1)[:, None])
        return self.seq_head(pooled)
