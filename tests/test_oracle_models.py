"""Pins of the oracle's model forwards and of the merged run (concatenate,
pad, run once, split): identity-model routing, row tags, NaN padding that
must never leak, batched == unbatched bit for bit, the ranking input layout
with one-hot tables, and the closed forms of masked mean pooling."""
import numpy as np
import pytest

import synth
from oracle import batching as ob
from oracle import models as om
from oracle import numerics as nx
from synth import Layer, Model, Params, Payload


def _rand_params(model, seed, tables_scale=0.125):
    rng = np.random.default_rng(seed)
    ws = [(rng.standard_normal((L.fan_out, L.fan_in)).astype(np.float32) / np.sqrt(L.fan_in),
           rng.uniform(-0.5, 0.5, L.fan_out).astype(np.float32)) for L in model.layers]
    tables = [(rng.standard_normal((model.table_rows, model.emb_dim)) * tables_scale).astype(np.float32)
              for _ in range(model.n_tables)]
    head = None
    if model.head is not None:
        head = (rng.standard_normal((model.head.fan_out, model.head.fan_in)).astype(np.float32) / 16,
                rng.uniform(-0.5, 0.5, model.head.fan_out).astype(np.float32))
    return Params(ws, tables, head)


MLP32 = Model(kind="mlp", dtype="f32", seed_id=0, layers=(Layer(12, 20, "relu"), Layer(20, 5, "none")))
MLP16 = Model(kind="mlp", dtype="bf16", seed_id=0, layers=(Layer(16, 24, "relu"), Layer(24, 8, "none")))
RANK = Model(kind="ranking", dtype="bf16", seed_id=0,
             layers=(Layer(4 * 8 + 3, 16, "relu"), Layer(16, 1, "sigmoid")),
             n_tables=4, table_rows=50, emb_dim=8, n_dense=3, bag_len=(1, 5))
SEQ = Model(kind="seqpool", dtype="f32", seed_id=0, layers=(Layer(6, 10, "relu"), Layer(10, 6, "none")),
            head=Layer(6, 2, "softmax"))


def _payloads(model, n_rows, rng, seq_max=9):
    out = []
    for n in n_rows:
        if model.kind == "mlp":
            out.append(Payload(rng.standard_normal((n, model.d_in)).astype(np.float32)))
        elif model.kind == "ranking":
            lens = rng.integers(0, 6, size=(n, model.n_tables)).astype(np.int32)
            ids = rng.integers(0, model.table_rows, size=int(lens.sum())).astype(np.int32)
            out.append(Payload(rng.standard_normal((n, model.n_dense)).astype(np.float32), lens, ids))
        else:
            L = rng.integers(1, seq_max + 1, size=n).astype(np.int32)
            out.append(Payload(rng.standard_normal((int(L.sum()), model.d_in)).astype(np.float32), L))
    return out


def test_identity_model_routes_rows_exactly():
    d = 6
    m = Model(kind="mlp", dtype="f32", seed_id=0, layers=(Layer(d, d, "none"),))
    p = Params([(np.eye(d, dtype=np.float32), np.zeros(d, np.float32))], [])
    o = om.OracleModel(m, p)
    # row tags: row i of request r holds (r, i, r*100+i, ...)
    n_rows = [3, 1, 4, 2]
    pays = []
    for r, n in enumerate(n_rows):
        x = np.zeros((n, d), np.float32)
        x[:, 0] = r
        x[:, 1] = np.arange(n)
        x[:, 2] = r * 100 + np.arange(n)
        pays.append(Payload(x))
    outs = ob.run_batch(o, pays, 16, pad=np.nan)
    for r, (y, pl) in enumerate(zip(outs, pays)):
        assert np.array_equal(y, pl.dense)


@pytest.mark.parametrize("model", [MLP32, MLP16, RANK, SEQ], ids=["mlp32", "mlp16", "ranking", "seqpool"])
@pytest.mark.parametrize("pad", [0.0, np.nan])
def test_batched_equals_unbatched_bitwise(model, pad):
    rng = np.random.default_rng(11)
    o = om.OracleModel(model, _rand_params(model, 3))
    n_rows = rng.integers(1, 6, size=7).tolist()
    pays = _payloads(model, n_rows, rng)
    P = sum(n_rows) + 5
    outs = ob.run_batch(o, pays, P, pad=pad, bucket_len=9)
    for y, pl in zip(outs, pays):
        ref = o.forward(pl)
        assert not np.isnan(y).any()
        assert np.array_equal(y, ref)
        assert y.shape[0] == (pl.lens.shape[0] if model.kind == "seqpool" else pl.dense.shape[0])


def test_ranking_input_layout_one_hot():
    # table f row i = (f + 1) * e_{i mod 8}: slot 8f+k of a row counts bag (e, f)'s
    # ids with id mod 8 == k, times f + 1; dense features follow the 4 pools
    m = RANK
    tables = []
    for f in range(m.n_tables):
        T = np.zeros((m.table_rows, m.emb_dim), np.float32)
        T[np.arange(m.table_rows), np.arange(m.table_rows) % 8] = f + 1
        tables.append(T)
    p = _rand_params(m, 0)
    p.tables = tables
    o = om.OracleModel(m, p)
    rng = np.random.default_rng(5)
    n = 6
    lens = rng.integers(0, 6, size=(n, m.n_tables)).astype(np.int32)
    ids = rng.integers(0, m.table_rows, size=int(lens.sum())).astype(np.int32)
    dense = np.array(rng.standard_normal((n, m.n_dense)), np.float32)
    X = o.ranking_input(dense, lens, ids)
    pos = 0
    for e in range(n):
        for f in range(m.n_tables):
            bag = ids[pos:pos + lens[e, f]]
            pos += lens[e, f]
            hist = np.bincount(bag % 8, minlength=8) * (f + 1)
            assert np.array_equal(X[e, 8 * f:8 * f + 8], hist)
        assert np.array_equal(X[e, 32:], nx.round_bf16(dense[e]))


def test_seqpool_constant_sequence_and_single_token():
    m = SEQ
    o = om.OracleModel(m, _rand_params(m, 9))
    tok = np.random.default_rng(2).standard_normal((1, m.d_in)).astype(np.float32)
    one = o.forward(Payload(tok, np.array([1], np.int32)))
    # L identical tokens: the mean is that token's MLP output exactly
    for L in (2, 7, 512):
        y = o.forward(Payload(np.repeat(tok, L, axis=0), np.array([L], np.int32)))
        assert np.array_equal(y, one)
    # L = 1 reduces to the unpooled MLP followed by the head
    h = o.mlp(nx.round_f32(tok))
    assert np.array_equal(one, o.seq_head(h).astype(np.float32))
    # equal logits give (0.5, 0.5)
    p = _rand_params(m, 9)
    p.head = (np.zeros((2, m.d_in), np.float32), np.array([0.3, 0.3], np.float32))
    assert np.array_equal(om.OracleModel(m, p).forward(Payload(tok, np.array([1], np.int32))), [[0.5, 0.5]])


def test_bf16_model_rounds_inputs():
    # a bf16 model sees bf16 inputs: x and round_bf16(x) give the same output
    o = om.OracleModel(MLP16, _rand_params(MLP16, 4))
    x = np.random.default_rng(3).standard_normal((5, 16)).astype(np.float32)
    y1 = o.forward(Payload(x))
    y2 = o.forward(Payload(nx.round_bf16(x).astype(np.float32)))
    assert np.array_equal(y1, y2)


def _golden_model(g, dtype):
    W1, W2 = np.array(g["W1"], np.float32), np.array(g["W2"], np.float32)
    m = Model(kind="mlp", dtype=dtype, seed_id=0,
              layers=(Layer(W1.shape[1], W1.shape[0], g["act1"]), Layer(W2.shape[1], W2.shape[0], g["act2"])))
    p = Params([(W1, np.array(g["b1"], np.float32)), (W2, np.array(g["b2"], np.float32))], [])
    return om.OracleModel(m, p)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_model_storage_rounding_chain_hand_worked(golden_dir, dtype):
    # every storage rounding of the model's forward (inputs, weights, biases,
    # hidden outputs, last output) against exact hand arithmetic; the golden
    # lists the value each plausible misplaced rounding would give instead
    import json
    import os
    g = json.load(open(os.path.join(golden_dir, f"mlp_rounding_{dtype}.json")))
    o = _golden_model(g, dtype)
    y = o.forward(Payload(np.array([g["x"]], np.float32)))
    assert y.dtype == np.float32
    assert y.tolist() == [g["y"]], (y.tolist(), g["y"])
    # the ranking and sequence models run the same layer chain
    assert np.array_equal(o.mlp(o._round_in(np.array([g["x"]], np.float32))).astype(np.float32), y)


def test_workload_models_build_and_run():
    # every workload's servables run on their first request
    for name in ("small_mlp", "multi_tenant", "ragged_seq"):
        w = synth.workload(name)
        t = synth.trace(w, 40)
        for r in range(40):
            s = int(t.servable[r])
            if w.models[s].kind == "ranking":
                continue
            o = om.OracleModel(w.models[s], synth.model_params(w, s))
            y = o.forward(synth.request_payload(t, r))
            assert y.shape == (int(t.n_rows[r]), w.models[s].d_out)
            assert np.isfinite(y).all()
            break
