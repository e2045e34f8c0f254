"""GPU parity of each kernel of the batching path against the oracle, called
through the C ABI (rb_k_*), on shapes that span several tiles, ragged tails
and padding. Bit-exact for routing and copies; the floating-point kernels are
held to the oracle's fp64 result within the stated tolerances."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import batching as ob
from oracle import numerics as nx
from paper_1712_06139_amd import rb

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _stream():
    return rb.torch_stream_ptr()


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _err():
    return torch.zeros(1, dtype=torch.int32, device=DEV)


def _rows_np(t):
    return t.cpu().numpy().view(np.uint8).view(rb.K_ROW_DTYPE)


def _make_group(rng, kind, n_batches, B, allowed, d_in, d_out, n_tables=0, seq_T=0, max_n=None, lens_gen=None):
    """Random batches of requests laid out like a trace arena. lens_gen(rng,
    n, n_tables) draws the bag lengths of ranking requests (default 0..20)."""
    max_n = max_n or B
    batches, reqs = [], []
    dense, lens, ids = [], [], []
    dense_off = lens_off = ids_off = out_off = 0
    row_base = 0
    for _ in range(n_batches):
        s, nreq, begin = 0, 0, len(reqs)
        while True:
            n = int(rng.integers(1, max_n + 1))
            if s + n > B or (nreq and rng.random() < 0.1):
                break
            if kind == rb.RB_MODEL_SEQPOOL:
                L = rng.integers(1, seq_T + 1, size=n)
                d = rng.standard_normal((int(L.sum()), d_in)).astype(np.float32)
                ln = L.astype(np.int32)
                ii = np.zeros(0, np.int32)
            elif kind == rb.RB_MODEL_RANKING:
                d = rng.standard_normal((n, d_in)).astype(np.float32)
                ln = (lens_gen(rng, n, n_tables) if lens_gen else rng.integers(0, 21, size=(n, n_tables))).astype(np.int32)
                ii = rng.integers(0, 1000, size=int(ln.sum())).astype(np.int32)
            else:
                d = rng.standard_normal((n, d_in)).astype(np.float32)
                ln = np.zeros(0, np.int32)
                ii = np.zeros(0, np.int32)
            reqs.append((dense_off, dense_off + d.size, lens_off, ids_off, ids_off + ii.size, out_off, n))
            dense.append(d.ravel()); lens.append(ln.ravel()); ids.append(ii)
            dense_off += d.size; lens_off += ln.size; ids_off += ii.size; out_off += n * d_out
            s += n
            nreq += 1
        P = ob.padded_size(s, allowed)
        batches.append((begin, nreq, row_base, P, s, seq_T))
        row_base += P
    kb = np.array(batches, dtype=np.int32).view(rb.K_BATCH_DTYPE).ravel()
    kr = np.zeros(len(reqs), dtype=rb.K_REQ_DTYPE)
    tok = 0  # seqpool: each request's first row among the group's packed tokens
    for i, r in enumerate(reqs):
        kr[i] = r + (tok,)
        if kind == rb.RB_MODEL_SEQPOOL:
            tok += (r[1] - r[0]) // d_in
    arena = dict(dense=np.concatenate(dense), lens=np.concatenate(lens) if lens_off else np.zeros(1, np.int32),
                 ids=np.concatenate(ids) if ids_off else np.zeros(1, np.int32), out_len=out_off)
    return kb, kr, arena, row_base


def _route(kind, kb, kr, arena, rows_total, d_in, d_out, n_tables=0):
    rows = torch.empty(rows_total * 4, dtype=torch.int64, device=DEV)
    err = _err()
    # device tensors stay referenced until the kernel has run
    lens = _dev(arena["lens"])
    kb_d = _dev(kb.view(np.uint8))
    kr_d = _dev(kr.view(np.uint8))
    rb.check(rb.lib().rb_k_route(_stream(), kind, rb.dptr(kb_d), len(kb), rb.dptr(kr_d), len(kr), rb.dptr(lens),
                                 int(arena["lens"].size), d_in, d_out, n_tables, rb.dptr(rows), rows_total,
                                 int(arena["out_len"]), rb.dptr(err)), "rb_k_route")
    torch.cuda.synchronize()
    return rows, err


def _expected_rows(kind, kb, kr, arena, d_in, d_out, n_tables=0):
    """Row map from the oracle's routing (exclusive prefix sums)."""
    out = []
    for b in kb:
        rq = kr[b["req_begin"]:b["req_begin"] + b["n_req"]]
        dst = ob.dst_rows(rq["n_rows"])
        rows = [(-1, 0, -1, -1)] * int(b["padded"])
        for q, d0 in zip(rq, dst):
            n = int(q["n_rows"])
            if kind == rb.RB_MODEL_SEQPOOL:
                L = arena["lens"][q["lens_off"]:q["lens_off"] + n]
                t0 = np.concatenate([[0], np.cumsum(L)[:-1]])
                for e in range(n):
                    rows[d0 + e] = (q["dense_off"] + t0[e] * d_in, int(L[e]), q["tok_off"] + t0[e],
                                    q["out_off"] + e * d_out)
            else:
                id0 = q["ids_off"]
                for e in range(n):
                    lo = q["lens_off"] + e * n_tables if kind == rb.RB_MODEL_RANKING else -1
                    rows[d0 + e] = (q["dense_off"] + e * d_in, id0, lo, q["out_off"] + e * d_out)
                    if kind == rb.RB_MODEL_RANKING:
                        id0 += int(arena["lens"][lo:lo + n_tables].sum())
        out.extend(rows)
    return np.array(out, dtype=np.int64)


@pytest.mark.parametrize("kind,B,allowed,d_in,d_out,nt,T", [
    (rb.RB_MODEL_MLP, 32, (8, 16, 32), 64, 16, 0, 0),
    (rb.RB_MODEL_MLP, 1024, (128, 256, 512, 1024), 40, 7, 0, 0),
    (rb.RB_MODEL_RANKING, 512, (64, 128, 256, 512), 13, 1, 26, 0),
    (rb.RB_MODEL_SEQPOOL, 64, (), 16, 2, 0, 64),
])
def test_route_bit_exact(kind, B, allowed, d_in, d_out, nt, T):
    rng = np.random.default_rng(1)
    kb, kr, arena, R = _make_group(rng, kind, 7, B, allowed, d_in, d_out, nt, T,
                                   max_n=64 if kind == rb.RB_MODEL_RANKING else (4 if T else 32))
    rows, err = _route(kind, kb, kr, arena, R, d_in, d_out, nt)
    got = _rows_np(rows)
    want = _expected_rows(kind, kb, kr, arena, d_in, d_out, nt)
    assert int(err.item()) == 0
    g = np.stack([got["src"], got["aux"], got["lens"], got["out"]], axis=1)
    pad = want[:, 0] < 0
    assert np.array_equal(g[~pad], want[~pad])
    assert np.all(g[pad][:, 0] == -1) and np.all(g[pad][:, 3] == -1)


@pytest.mark.parametrize("bf16", [0, 1])
@pytest.mark.parametrize("d_in,ldx", [(64, 64), (4096, 4096), (13, 64), (40, 64), (40, 72), (100, 200)])
def test_assemble_bit_exact(bf16, d_in, ldx):
    rng = np.random.default_rng(2)
    kb, kr, arena, R = _make_group(rng, rb.RB_MODEL_MLP, 5, 256, (64, 128, 256), d_in, 4, max_n=32)
    rows, err = _route(rb.RB_MODEL_MLP, kb, kr, arena, R, d_in, 4)
    dense = _dev(arena["dense"])
    X = torch.empty((R, ldx), dtype=torch.int16 if bf16 else torch.float32, device=DEV)
    rb.check(rb.lib().rb_k_assemble(_stream(), rb.dptr(rows), R, 0, 0, rb.dptr(dense), dense.numel(), d_in,
                                    rb.dptr(X), ldx, bf16, float("nan"), rb.dptr(err)), "rb_k_assemble")
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    got = X.cpu().numpy()
    if bf16:
        got = (got.astype(np.uint16).astype(np.uint32) << 16).view(np.float32)
    for b in kb:
        rq = kr[b["req_begin"]:b["req_begin"] + b["n_req"]]
        pays = [synth_payload(arena["dense"][q["dense_off"]:q["dense_end"]].reshape(-1, d_in)) for q in rq]
        ref = ob.assemble(_MlpShape(d_in), pays, int(b["padded"]), pad=np.nan).dense
        if bf16:
            ref = nx.round_bf16(ref)
        blk = got[b["row_base"]:b["row_base"] + b["padded"]]
        assert np.array_equal(blk[:, :d_in], ref, equal_nan=True)
        assert np.all(blk[:, d_in:] == 0)


@pytest.mark.parametrize("T,ldx", [(64, 16), (48, 24), (128, 16)])
def test_assemble_seq_packed_bit_exact(T, ldx):
    # packed tokens: the real tokens of every sequence of the group in
    # consecutive rows (request order, then sequence order), nothing else written
    rng = np.random.default_rng(6)
    d_in = 16
    kb, kr, arena, R = _make_group(rng, rb.RB_MODEL_SEQPOOL, 5, 16, (8, 16), d_in, 2, 0, T, max_n=4)
    rows, err = _route(rb.RB_MODEL_SEQPOOL, kb, kr, arena, R, d_in, 2)
    dense = _dev(arena["dense"])
    M = R * T
    X = torch.full((M, ldx), -3.0, dtype=torch.float32, device=DEV)
    rb.check(rb.lib().rb_k_assemble(_stream(), rb.dptr(rows), M, T, 2, rb.dptr(dense), dense.numel(), d_in,
                                    rb.dptr(X), ldx, 0, float("nan"), rb.dptr(err)), "rb_k_assemble")
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    got = X.cpu().numpy()
    n_tok = int(sum((q["dense_end"] - q["dense_off"]) // d_in for q in kr))
    want = np.concatenate([arena["dense"][q["dense_off"]:q["dense_end"]].reshape(-1, d_in) for b in kb
                           for q in kr[b["req_begin"]:b["req_begin"] + b["n_req"]]])
    assert want.shape[0] == n_tok
    assert np.array_equal(got[:n_tok, :d_in], want)
    assert np.all(got[:n_tok, d_in:] == 0)
    assert np.all(got[n_tok:] == -3.0)
    # a packed row past the arena is reported, and nothing is written for it
    r_np = _rows_np(rows).copy()
    live = np.flatnonzero(r_np["src"] >= 0)
    r_np["lens"][live[-1]] = M - 1
    rows_bad = _dev(r_np.view(np.uint8))
    err2 = _err()
    X2 = torch.full((M, ldx), -3.0, dtype=torch.float32, device=DEV)
    rb.check(rb.lib().rb_k_assemble(_stream(), rb.dptr(rows_bad), M, T, 2, rb.dptr(dense), dense.numel(), d_in,
                                    rb.dptr(X2), ldx, 0, 0.0, rb.dptr(err2)), "rb_k_assemble")
    torch.cuda.synchronize()
    L_last = int(r_np["aux"][live[-1]])
    assert int(err2.item()) == (1 if L_last > 1 else 0)
    assert np.all(X2.cpu().numpy()[M - 1, :d_in] == (-3.0 if L_last > 1 else want[-1]))


@pytest.mark.parametrize("T,ldx,skip", [(64, 16, 0), (48, 16, 0), (64, 24, 0), (128, 16, 0), (128, 16, 1),
                                         (192, 24, 1)])
def test_assemble_seq_bit_exact(T, ldx, skip):
    # sequences padded along time to T: token t < L of slot e at row e*T + t,
    # pad value elsewhere (power-of-two and general index paths); with
    # real-only, rows t >= L and padding slots stay untouched
    rng = np.random.default_rng(5)
    d_in = 16
    kb, kr, arena, R = _make_group(rng, rb.RB_MODEL_SEQPOOL, 5, 16, (8, 16), d_in, 2, 0, T, max_n=4)
    rows, err = _route(rb.RB_MODEL_SEQPOOL, kb, kr, arena, R, d_in, 2)
    dense = _dev(arena["dense"])
    M = R * T
    X = torch.full((M, ldx), -3.0, dtype=torch.float32, device=DEV)
    rb.check(rb.lib().rb_k_assemble(_stream(), rb.dptr(rows), M, T, skip, rb.dptr(dense), dense.numel(), d_in,
                                    rb.dptr(X), ldx, 0, float("nan"), rb.dptr(err)), "rb_k_assemble")
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    got = X.cpu().numpy().reshape(R, T, ldx)
    from synth import Payload
    for b in kb:
        rq = kr[b["req_begin"]:b["req_begin"] + b["n_req"]]
        pays = [Payload(arena["dense"][q["dense_off"]:q["dense_end"]],
                        arena["lens"][q["lens_off"]:q["lens_off"] + q["n_rows"]]) for q in rq]
        asm = ob.assemble(_SeqShape(d_in), pays, int(b["padded"]), pad=np.nan, bucket_len=T)
        ref = asm.tokens
        blk = got[b["row_base"]:b["row_base"] + b["padded"]]
        if skip:
            live = np.arange(T)[None, :] < asm.seq_len[:, None]  # pad slots have L = 0
            assert np.array_equal(blk[live][:, :d_in], ref[live], equal_nan=True)
            assert np.all(blk[live][:, d_in:] == 0)
            assert np.all(blk[~live] == -3.0)
            assert (~live).any()
        else:
            assert np.array_equal(blk[:, :, :d_in], ref, equal_nan=True)
            assert np.all(blk[:, :, d_in:] == 0)
    # real-only needs a sequence layout
    assert rb.lib().rb_k_assemble(_stream(), rb.dptr(rows), M, 0, 1, rb.dptr(dense), dense.numel(),
                                  d_in, rb.dptr(X), ldx, 0, 0.0, rb.dptr(err)) == rb.RB_EINVAL


class _SeqShape:
    kind = "seqpool"

    def __init__(self, d_in):
        self.d_in = d_in


class _MlpShape:
    kind = "mlp"

    def __init__(self, d_in):
        self.d_in = d_in


def synth_payload(d):
    from synth import Payload
    return Payload(d)


def _lens_skewed(rng, n, nt):
    # mostly empty bags, now and then one long bag (many chunks of 8 ids)
    ln = rng.integers(0, 2, size=(n, nt)) * (rng.random((n, nt)) < 0.2)
    long = rng.random(n) < 0.3
    ln[long, rng.integers(0, nt, size=int(long.sum()))] = rng.integers(30, 700, size=int(long.sum()))
    return ln


_LENS = {
    "uniform": None,                                            # 0..20 per bag
    "tiny": lambda rng, n, nt: rng.integers(0, 2, size=(n, nt)),  # rows with fewer ids than lane groups
    "skewed": _lens_skewed,
    "all_empty": lambda rng, n, nt: np.zeros((n, nt), np.int64),
}


@pytest.mark.parametrize("entry", ["rb_k_embbag", "rb_k_embbag_dedup"])
@pytest.mark.parametrize("lens,nt", [(k, 26) for k in _LENS] + [("uniform", 1), ("uniform", 5), ("uniform", 64)])
def test_embbag_matches_oracle(lens, nt, entry):
    # 26 tables (the ranking model) with every bag-length mix, and 1, 5 and 64
    # tables (the most a row may have): a bag's start is the sum of the lengths
    # of the row's earlier bags, loaded up to 8 per lane
    rng = np.random.default_rng(3)
    rows_t = 1000
    kb, kr, arena, R = _make_group(rng, rb.RB_MODEL_RANKING, 4, 512, (64, 128, 256, 512), 13, 1, nt, 0,
                                   max_n=64, lens_gen=_LENS[lens])
    rows, err = _route(rb.RB_MODEL_RANKING, kb, kr, arena, R, 13, 1, nt)
    tables = [(rng.standard_normal((rows_t, 64)) / 8).astype(np.float32) for _ in range(nt)]
    tb = [nx.round_bf16(t).astype(np.float32) for t in tables]
    dev_t = [torch.from_numpy((t.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).to(DEV) for t in tb]
    ptrs = _dev(np.array([t.data_ptr() for t in dev_t], dtype=np.uint64).view(np.int64))
    ldx = (nt * 64 + 13 + 63) // 64 * 64
    X = torch.empty((R, ldx), dtype=torch.int16, device=DEV)
    dense, lens, ids = _dev(arena["dense"]), _dev(arena["lens"]), _dev(arena["ids"])
    rb.check(getattr(rb.lib(), entry)(_stream(), rb.dptr(rows), R, rb.dptr(lens), rb.dptr(ids), ids.numel(),
                                      rb.dptr(ptrs), nt, rows_t, 64, rb.dptr(dense), 13, rb.dptr(X), ldx, 0.0,
                                      rb.dptr(err)), entry)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    got = (X.cpu().numpy().astype(np.uint16).astype(np.uint32) << 16).view(np.float32)
    rmap = _rows_np(rows)
    from oracle.models import OracleModel
    from synth import Layer, Model, Params
    m = Model(kind="ranking", dtype="bf16", seed_id=0, layers=(Layer(nt * 64 + 13, 1, "sigmoid"),),
              n_tables=nt, table_rows=rows_t, emb_dim=64, n_dense=13)
    om = OracleModel(m, Params([(np.zeros((1, nt * 64 + 13), np.float32), np.zeros(1, np.float32))], tables))
    om_abs = OracleModel(m, Params([(np.zeros((1, nt * 64 + 13), np.float32), np.zeros(1, np.float32))],
                                   [np.abs(t) for t in tb]))
    n_exact = n_tot = 0
    for r in range(R):
        rw = rmap[r]
        if rw["src"] < 0:
            assert np.all(got[r, :nt * 64 + 13] == 0) and np.all(got[r, nt * 64 + 13:] == 0)
            continue
        ln = arena["lens"][rw["lens"]:rw["lens"] + nt]
        ii = arena["ids"][rw["aux"]:rw["aux"] + ln.sum()]
        dn = arena["dense"][rw["src"]:rw["src"] + 13]
        ref = om.ranking_input(dn[None, :], ln[None, :], ii)[0]
        g = got[r, :nt * 64 + 13].astype(np.float64)
        # fp32 summation of n terms is within (n - 1) 2^-24 sum|x| of the exact
        # sum to first order (any order); bf16 rounding then adds at most one
        # bf16 ulp. The factor 2 covers the exact bound's second-order term and
        # an ulp taken at the oracle's value rather than the larger of the two
        sabs = om_abs.ranking_input(dn[None, :], ln[None, :], ii)[0]
        nterm = np.concatenate([np.repeat(np.maximum(ln - 1, 0), 64), np.zeros(13)])
        ulp = np.maximum(np.abs(ref), 2.0 ** -126) * 2.0 ** -7
        assert np.all(np.abs(g - ref) <= ulp + 2.0 * nterm * 2.0 ** -24 * sabs), r
        assert np.all(got[r, nt * 64 + 13:] == 0)
        n_exact += int(np.sum(g == ref))
        n_tot += g.size
    assert n_exact >= 0.99 * n_tot


@pytest.mark.parametrize("entry", ["rb_k_embbag", "rb_k_embbag_dedup"])
@pytest.mark.parametrize("cut", [1, 13, 31, 45])
def test_embbag_ragged_row_count_and_pad_value(cut, entry):
    # a row count that leaves the last row block part empty (groups with no
    # bag) and a non-zero pad: real rows are bit-identical to the full call,
    # padding rows hold pad in every bag and dense-feature column and zeros in
    # the tail, and rows past the count are not written
    rng = np.random.default_rng(29)
    nt, rows_t = 26, 1000
    kb, kr, arena, R = _make_group(rng, rb.RB_MODEL_RANKING, 4, 512, (64, 128, 256, 512), 13, 1, nt, 0,
                                   max_n=64, lens_gen=None)
    rows, _ = _route(rb.RB_MODEL_RANKING, kb, kr, arena, R, 13, 1, nt)
    dev_t = [torch.randn(rows_t, 64, device=DEV).to(torch.bfloat16).view(torch.int16) for _ in range(nt)]
    ptrs = _dev(np.array([t.data_ptr() for t in dev_t], dtype=np.uint64).view(np.int64))
    dense, lens_d, ids = _dev(arena["dense"]), _dev(arena["lens"]), _dev(arena["ids"])
    outs = []
    for n, pad in ((R, 0.0), (R - cut, 1.5)):
        X = torch.full((R, 1728), 0x7FC1, dtype=torch.int16, device=DEV)
        err = _err()
        rb.check(getattr(rb.lib(), entry)(_stream(), rb.dptr(rows), n, rb.dptr(lens_d), rb.dptr(ids), ids.numel(),
                                          rb.dptr(ptrs), nt, rows_t, 64, rb.dptr(dense), 13, rb.dptr(X), 1728,
                                          pad, rb.dptr(err)), entry)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        outs.append(X.cpu().numpy())
    full, part = outs
    src = _rows_np(rows)["src"]
    n = R - cut
    real = src[:n] >= 0
    assert (~real).any() and real.any()
    assert np.array_equal(part[:n][real], full[:n][real])
    pad_bits = np.int16(0x3FC0)  # 1.5 in bf16
    assert np.all(part[:n][~real][:, :nt * 64 + 13] == pad_bits)
    assert np.all(part[:n][~real][:, nt * 64 + 13:] == 0)
    assert np.all(part[n:] == np.int16(0x7FC1))


@pytest.mark.parametrize("lens", list(_LENS))
@pytest.mark.parametrize("ids_kind", ["zipf", "uniform", "invalid"])
def test_embbag_dedup_bit_identical(lens, ids_kind):
    # the per-block dedup of ids changes which table rows are gathered, not the
    # sums: every bag is added in id order in fp32 either way, so both kernels
    # give the same bits (and the same error flag). Zipf ids (few distinct per
    # block), uniform ids over a small table (more distinct rows than the LDS
    # holds), and ids outside their table
    rng = np.random.default_rng(17)
    nt, rows_t = 26, 1000 if ids_kind == "uniform" else 100_000
    kb, kr, arena, R = _make_group(rng, rb.RB_MODEL_RANKING, 5, 512, (64, 128, 256, 512), 13, 1, nt, 0,
                                   max_n=64, lens_gen=_LENS[lens])
    n_ids = arena["ids"].size
    if ids_kind != "uniform" and n_ids > 1:
        # Zipf(1.1) ranks through a fixed permutation of the table rows
        z = np.minimum(rng.zipf(1.1, size=n_ids), rows_t) - 1
        arena["ids"][:] = rng.permutation(rows_t)[z].astype(np.int32)
    if ids_kind == "invalid" and n_ids > 3:
        arena["ids"][[0, n_ids // 2, n_ids - 1]] = [rows_t, -5, rows_t + 123]
    rows, err0 = _route(rb.RB_MODEL_RANKING, kb, kr, arena, R, 13, 1, nt)
    dev_t = [torch.randn(rows_t, 64, device=DEV).to(torch.bfloat16).view(torch.int16) for _ in range(nt)]
    ptrs = _dev(np.array([t.data_ptr() for t in dev_t], dtype=np.uint64).view(np.int64))
    dense, lens_d, ids = _dev(arena["dense"]), _dev(arena["lens"]), _dev(arena["ids"])
    outs, errs = [], []
    for entry in ("rb_k_embbag", "rb_k_embbag_dedup"):
        X = torch.full((R, 1728), 0x7FC1, dtype=torch.int16, device=DEV)
        err = _err()
        rb.check(getattr(rb.lib(), entry)(_stream(), rb.dptr(rows), R, rb.dptr(lens_d), rb.dptr(ids), ids.numel(),
                                          rb.dptr(ptrs), nt, rows_t, 64, rb.dptr(dense), 13, rb.dptr(X), 1728,
                                          0.0, rb.dptr(err)), entry)
        torch.cuda.synchronize()
        outs.append(X.cpu().numpy())
        errs.append(int(err.item()))
    assert np.array_equal(outs[0], outs[1])
    assert errs[0] == errs[1] == (1 if (ids_kind == "invalid" and n_ids > 3) else 0)


def _bf16_dev(a):
    b = nx.round_bf16(a).astype(np.float32)
    return torch.from_numpy((b.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).to(DEV), b


def _row_scaled_err(y, ref):
    scale = np.maximum(np.max(np.abs(ref), axis=1, keepdims=True), 1e-30)
    return np.max(np.abs(y - ref) / scale)


@pytest.mark.parametrize("M,N,K,act,out_f32,pad_y", [
    (1, 128, 64, rb.RB_ACT_NONE, 1, 0), (200, 256, 1728, rb.RB_ACT_RELU, 0, 0), (1024, 1024, 512, rb.RB_ACT_RELU, 0, 0),
    (333, 512, 1024, rb.RB_ACT_NONE, 1, 0), (130, 128, 4096, rb.RB_ACT_SIGMOID, 1, 0),
    (77, 256, 128, rb.RB_ACT_RELU, 0, 8), (300, 384, 256, rb.RB_ACT_NONE, 1, 24),
    # more tiles than compute units: 256 x 256 tiles of 8 waves with 2 stages
    # (XCD and plain tile order; K = 192, an odd number of k-steps), a
    # persistent grid of 256 x 128 tiles, ragged last rows
    (4500, 4096, 512, rb.RB_ACT_RELU, 0, 0), (4500, 4096, 192, rb.RB_ACT_NONE, 1, 8),
    (2100, 8192, 512, rb.RB_ACT_SIGMOID, 0, 0), (25600 - 37, 384, 192, rb.RB_ACT_RELU, 1, 0),
    # at least two 256 x 256 tiles per compute unit: 4 waves of 128 x 128 (XCD
    # and plain tile order)
    (8500, 4096, 192, rb.RB_ACT_RELU, 0, 0), (4500 + 11, 8192, 512, rb.RB_ACT_NONE, 1, 0),
    # few tiles: 128 x 128 when there are at least half as many as compute
    # units, else 128 x 64 (1024 x 1024), else 64 x 64 (the small shapes above)
    (2816 - 5, 1024, 1728, rb.RB_ACT_RELU, 0, 0), (2816 + 3, 512, 1024, rb.RB_ACT_SIGMOID, 1, 0)])
def test_gemm_bf16_matches_fp64(M, N, K, act, out_f32, pad_y):
    rng = np.random.default_rng(4)
    Xd, X = _bf16_dev(rng.standard_normal((M, K)))
    Wd, W = _bf16_dev(rng.standard_normal((N, K)) / np.sqrt(K))
    b = rng.uniform(-0.5, 0.5, N).astype(np.float32)
    bd = _dev(b)
    ldy = N + pad_y  # padded output rows: columns past N must stay untouched
    Y = torch.full((M, ldy), -7.0 if out_f32 else 0x5a5a, dtype=torch.float32 if out_f32 else torch.int16,
                   device=DEV)
    rb.check(rb.lib().rb_k_gemm_bf16(_stream(), rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(bd), rb.dptr(Y), ldy, M, N,
                                     K, act, out_f32), "gemm_bf16")
    torch.cuda.synchronize()
    full = Y.cpu().numpy()
    assert np.all(full[:, N:] == (-7.0 if out_f32 else 0x5a5a))
    got = full[:, :N]
    if not out_f32:
        got = (got.astype(np.uint16).astype(np.uint32) << 16).view(np.float32)
    name = {0: "none", 1: "relu", 2: "sigmoid"}[act]
    ref = nx.dense(X, W, b, name)
    # fp32 accumulation of exact bf16 products: far inside the 2e-2 bf16 bar
    tol = 2e-2 if not out_f32 else 1e-4
    assert _row_scaled_err(got, ref) <= tol
    if not out_f32:
        assert np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-3)) <= 2.0 ** -7
    # the output stride must keep 16-byte row alignment
    assert rb.lib().rb_k_gemm_bf16(_stream(), rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(bd), rb.dptr(Y), N + 4, M,
                                   N, K, act, out_f32) == rb.RB_EINVAL


@pytest.mark.parametrize("M,N,K,act", [(1, 64, 64, rb.RB_ACT_RELU), (257, 1024, 256, rb.RB_ACT_RELU),
                                       (1000, 64, 1024, rb.RB_ACT_NONE), (64 * 64, 512, 256, rb.RB_ACT_RELU),
                                       (300, 1024, 1088, rb.RB_ACT_SIGMOID), (70, 192, 32, rb.RB_ACT_RELU)])
def test_gemm_f32_matches_fp64(M, N, K, act):
    rng = np.random.default_rng(5)
    X = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32)
    b = rng.uniform(-0.5, 0.5, N).astype(np.float32)
    Y = torch.empty((M, N), dtype=torch.float32, device=DEV)
    Xd, Wd, bd = _dev(X), _dev(W), _dev(b)
    rb.check(rb.lib().rb_k_gemm_f32(_stream(), rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(bd),
                                    rb.dptr(Y), N, M, N, K, act, None, 0), "gemm_f32")
    torch.cuda.synchronize()
    ref = nx.dense(X, W, b, {rb.RB_ACT_NONE: "none", rb.RB_ACT_RELU: "relu", rb.RB_ACT_SIGMOID: "sigmoid"}[act])
    assert _row_scaled_err(Y.cpu().numpy(), ref) <= 1e-5


@pytest.mark.parametrize("dtype,N,K", [("f32", 512, 256), ("f32", 1024, 1088), ("bf16", 512, 256),
                                        ("bf16", 1024, 2112), ("bf16", 4096, 512), ("bf16", 2048, 1728)])
def test_gemm_rows_independent_of_batch(dtype, N, K):
    # a row's output bits do not depend on how many rows share the launch or on
    # where it sits among them: the same k order for every M, tile shape and
    # tile order (K = 1088 / 2112 / 1728 puts W above 4 MB: plain tile order; the
    # bf16 launch of all rows takes a larger tile than the partial ones: N = 4096
    # and 2048 give the full launch at least two 256 x 256 tiles per compute
    # unit (4 waves of 128 x 128, 2 stages),
    # while the partial launches take 128 x 64 or 64 x 64 tiles with 4 stages)
    rng = np.random.default_rng(11)
    M = 16384
    X = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32)
    b = rng.uniform(-0.5, 0.5, N).astype(np.float32)
    bd = _dev(b)
    if dtype == "f32":
        Xd, Wd = _dev(X), _dev(W)
        esz, call = 4, rb.lib().rb_k_gemm_f32
        extra = (None, 0)
    else:
        Xd, _ = _bf16_dev(X)
        Wd, _ = _bf16_dev(W)
        esz, call = 2, rb.lib().rb_k_gemm_bf16
        extra = (1,)
    Y = torch.empty((M, N), dtype=torch.float32, device=DEV)
    rb.check(call(_stream(), rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(bd), rb.dptr(Y), N, M, N, K,
                  rb.RB_ACT_RELU, *extra), "gemm")
    for r0, m in ((0, 1), (8191, 1), (M - 1, 1), (64, 300), (10257, 443)):
        Yp = torch.empty((m, N), dtype=torch.float32, device=DEV)
        rb.check(call(_stream(), rb.dptr(Xd) + r0 * K * esz, K, rb.dptr(Wd), K, rb.dptr(bd), rb.dptr(Yp), N, m,
                      N, K, rb.RB_ACT_RELU, *extra), "gemm")
        torch.cuda.synchronize()
        assert torch.equal(Yp, Y[r0:r0 + m]), (r0, m)


@pytest.mark.parametrize("T", [64, 128, 256])
def test_gemm_f32_skips_padding_token_blocks(T):
    # sequence layout: slot e owns rows [e*T, (e+1)*T); 64-row blocks at or past
    # the slot's length (and every block of a pad slot) are neither computed
    # nor stored; every block holding a real token matches fp64 in full
    rng = np.random.default_rng(7)
    n_slots, N, K = 9, 128, 64
    L = rng.integers(1, T + 1, size=n_slots)
    L[2] = T
    src = np.where(np.arange(n_slots) == 5, -1, 0)  # slot 5 is padding
    rows = _rows_dev(src, L, np.arange(n_slots))
    M = n_slots * T
    X = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32)
    b = rng.uniform(-0.5, 0.5, N).astype(np.float32)
    Y = torch.full((M, N), -7.0, dtype=torch.float32, device=DEV)
    Xd, Wd, bd = _dev(X), _dev(W), _dev(b)
    rb.check(rb.lib().rb_k_gemm_f32(_stream(), rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(bd), rb.dptr(Y), N, M, N,
                                    K, rb.RB_ACT_RELU, rb.dptr(rows), T), "gemm_f32")
    torch.cuda.synchronize()
    got = Y.cpu().numpy()
    ref = nx.dense(X, W, b, "relu")
    t = np.arange(M) % T
    e = np.arange(M) // T
    live = (src[e] >= 0) & ((t // 64) * 64 < L[e])
    assert _row_scaled_err(got[live], ref[live]) <= 1e-5
    assert np.all(got[~live] == -7.0)
    # bad skip_T is rejected
    assert rb.lib().rb_k_gemm_f32(_stream(), rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(bd), rb.dptr(Y), N, M, N, K,
                                  rb.RB_ACT_RELU, rb.dptr(rows), 48) == rb.RB_EINVAL


def _rows_dev(src, aux, out):
    a = np.zeros(len(src), dtype=rb.K_ROW_DTYPE)
    a["src"], a["aux"], a["lens"], a["out"] = src, aux, -1, out
    return _dev(a.view(np.uint8))


@pytest.mark.parametrize("K,ldh", [(256, 256), (264, 272), (100, 100), (1000, 1004)])
def test_head_and_split(K, ldh):
    # 16-byte path (K and ldh multiples of 8) and element path; rows whose
    # output is -1 are skipped
    rng = np.random.default_rng(6)
    R = 300
    out_idx = np.where(rng.random(R) < 0.8, np.arange(R) * 3, -1)
    rows = _rows_dev(np.zeros(R), np.zeros(R), out_idx)
    Hd, Hf = _bf16_dev(rng.standard_normal((R, ldh)))
    H = Hf[:, :K]
    wd, w = _bf16_dev(rng.standard_normal(K) / 16)
    out = torch.full((R * 3,), -7.0, device=DEV)
    rb.check(rb.lib().rb_k_head(_stream(), rb.dptr(rows), R, rb.dptr(Hd), ldh, rb.dptr(wd), 0.25, K,
                                rb.RB_ACT_SIGMOID, rb.dptr(out)), "head")
    Y = rng.standard_normal((R, 64)).astype(np.float32)
    out2 = torch.full((R * 3 * 10,), -7.0, device=DEV)
    rows2 = _rows_dev(np.zeros(R), np.zeros(R), np.where(out_idx >= 0, out_idx * 10, -1))
    Yd = _dev(Y)
    rb.check(rb.lib().rb_k_split(_stream(), rb.dptr(rows2), R, rb.dptr(Yd), 64, 30, rb.dptr(out2)), "split")
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    o2 = out2.cpu().numpy()
    ref = nx.sigmoid(H.astype(np.float64) @ w.astype(np.float64) + 0.25)
    for r in range(R):
        if out_idx[r] < 0:
            continue
        assert abs(o[out_idx[r]] - ref[r]) <= 1e-5 * abs(ref[r])
        assert np.array_equal(o2[out_idx[r] * 10:out_idx[r] * 10 + 30], Y[r, :30])
    keep = np.zeros(R * 3, bool)
    keep[out_idx[out_idx >= 0]] = True
    assert np.all(o[~keep] == -7.0)


@pytest.mark.parametrize("M,K2,act", [(1, 1024, rb.RB_ACT_SIGMOID), (77, 1024, rb.RB_ACT_SIGMOID),
                                       (128, 192, rb.RB_ACT_NONE), (300, 1024, rb.RB_ACT_SIGMOID),
                                       (4500, 1024, rb.RB_ACT_SIGMOID), (32768, 1024, rb.RB_ACT_SIGMOID)])
def test_mlp_tail_bit_identical_to_separate_kernels(M, K2, act):
    # the fused last two layers + head against rb_k_gemm_bf16 twice and
    # rb_k_head on the same operands: the same bits in every output, rows
    # whose output is -1 skipped, ragged last blocks; and within the fp64
    # bound of the definition
    rng = np.random.default_rng(23)
    ldh = K2 + 64
    H1d, H1 = _bf16_dev(np.maximum(rng.standard_normal((M, ldh)), 0))
    W2d, W2 = _bf16_dev(rng.standard_normal((512, K2)) / np.sqrt(K2))
    W3d, W3 = _bf16_dev(rng.standard_normal((256, 512)) / np.sqrt(512))
    w4d, w4 = _bf16_dev(rng.standard_normal(256) / 16)
    b2 = (rng.uniform(-0.5, 0.5, 512)).astype(np.float32)
    b3 = (rng.uniform(-0.5, 0.5, 256)).astype(np.float32)
    b2d, b3d = _dev(b2), _dev(b3)
    out_idx = np.where(rng.random(M) < 0.9, np.arange(M) * 2, -1)
    rows = _rows_dev(np.zeros(M), np.zeros(M), out_idx)
    st = _stream()
    Y2 = torch.empty((M, 512), dtype=torch.int16, device=DEV)
    Y3 = torch.empty((M, 256), dtype=torch.int16, device=DEV)
    ref = torch.full((M * 2,), -7.0, device=DEV)
    got = torch.full((M * 2,), -7.0, device=DEV)
    rb.check(rb.lib().rb_k_gemm_bf16(st, rb.dptr(H1d), ldh, rb.dptr(W2d), K2, rb.dptr(b2d), rb.dptr(Y2), 512, M, 512,
                                     K2, rb.RB_ACT_RELU, 0), "gemm 2")
    rb.check(rb.lib().rb_k_gemm_bf16(st, rb.dptr(Y2), 512, rb.dptr(W3d), 512, rb.dptr(b3d), rb.dptr(Y3), 256, M, 256,
                                     512, rb.RB_ACT_RELU, 0), "gemm 3")
    rb.check(rb.lib().rb_k_head(st, rb.dptr(rows), M, rb.dptr(Y3), 256, rb.dptr(w4d), 0.125, 256, act,
                                rb.dptr(ref)), "head")
    rb.check(rb.lib().rb_k_mlp_tail(st, rb.dptr(rows), M, rb.dptr(H1d), ldh, K2, rb.dptr(W2d), K2, rb.dptr(b2d),
                                    rb.dptr(W3d), 512, rb.dptr(b3d), rb.dptr(w4d), 0.125, act, rb.dptr(got)),
             "mlp_tail")
    torch.cuda.synchronize()
    g, r = got.cpu().numpy(), ref.cpu().numpy()
    assert np.array_equal(g, r)
    keep = np.zeros(M * 2, bool)
    keep[out_idx[out_idx >= 0]] = True
    assert np.all(g[~keep] == -7.0) and np.all(g[keep] != -7.0)
    # the definition in fp64 with the bf16 storage roundings, on a sample of rows
    sel = rng.choice(M, size=min(M, 64), replace=False)
    h = H1[sel, :K2].astype(np.float64)
    y2 = nx.round_bf16(np.maximum(h @ W2.astype(np.float64).T + b2, 0))
    y3 = nx.round_bf16(np.maximum(y2 @ W3.astype(np.float64).T + b3, 0))
    z = y3 @ w4.astype(np.float64) + 0.125
    want = nx.sigmoid(z) if act == rb.RB_ACT_SIGMOID else z
    for i, rr in enumerate(sel):
        if out_idx[rr] >= 0:
            assert abs(g[out_idx[rr]] - want[i]) <= 2e-2 * max(abs(want[i]), 1e-3), (rr, g[out_idx[rr]], want[i])


@pytest.mark.parametrize("M,K,act,hact", [(1000, 512, rb.RB_ACT_RELU, rb.RB_ACT_SIGMOID),
                                          (300, 192, rb.RB_ACT_RELU, rb.RB_ACT_NONE),
                                          (128, 64, rb.RB_ACT_NONE, rb.RB_ACT_SIGMOID),
                                          (4133, 512, rb.RB_ACT_RELU, rb.RB_ACT_SIGMOID),
                                          (20000 + 7, 512, rb.RB_ACT_RELU, rb.RB_ACT_SIGMOID)])
def test_gemm_head_bit_identical_to_separate_kernels(M, K, act, hact):
    # the last hidden layer (256 outputs) with the head in its epilogue against
    # rb_k_gemm_bf16 and rb_k_head on the same operands: the same bits in
    # every output, rows whose output is -1 skipped, ragged last tiles; and
    # within the fp64 bound of the definition. 64-row tiles below 128 x 128
    # rows (half the compute units' worth of 128-row tiles), 128-row tiles at
    # 20007 rows
    rng = np.random.default_rng(29)
    ldx = K + 64
    Xd, X = _bf16_dev(np.maximum(rng.standard_normal((M, ldx)), 0))
    Wd, W = _bf16_dev(rng.standard_normal((256, K)) / np.sqrt(K))
    wd, w = _bf16_dev(rng.standard_normal(256) / 16)
    b = rng.uniform(-0.5, 0.5, 256).astype(np.float32)
    bd = _dev(b)
    out_idx = np.where(rng.random(M) < 0.9, np.arange(M) * 2, -1)
    rows = _rows_dev(np.zeros(M), np.zeros(M), out_idx)
    st = _stream()
    Y = torch.empty((M, 256), dtype=torch.int16, device=DEV)
    ref = torch.full((M * 2,), -7.0, device=DEV)
    got = torch.full((M * 2,), -7.0, device=DEV)
    rb.check(rb.lib().rb_k_gemm_bf16(st, rb.dptr(Xd), ldx, rb.dptr(Wd), K, rb.dptr(bd), rb.dptr(Y), 256, M, 256, K,
                                     act, 0), "gemm")
    rb.check(rb.lib().rb_k_head(st, rb.dptr(rows), M, rb.dptr(Y), 256, rb.dptr(wd), 0.125, 256, hact, rb.dptr(ref)),
             "head")
    rb.check(rb.lib().rb_k_gemm_head(st, rb.dptr(Xd), ldx, rb.dptr(Wd), K, rb.dptr(bd), M, K, act, rb.dptr(rows),
                                     rb.dptr(wd), 0.125, hact, rb.dptr(got)), "gemm_head")
    torch.cuda.synchronize()
    g, r = got.cpu().numpy(), ref.cpu().numpy()
    assert np.array_equal(g, r)
    keep = np.zeros(M * 2, bool)
    keep[out_idx[out_idx >= 0]] = True
    assert np.all(g[~keep] == -7.0) and np.all(g[keep] != -7.0)
    # the definition in fp64 with the bf16 storage rounding, on a sample of rows
    sel = rng.choice(M, size=min(M, 64), replace=False)
    z = X[sel, :K].astype(np.float64) @ W.astype(np.float64).T + b
    y = nx.round_bf16(np.maximum(z, 0) if act == rb.RB_ACT_RELU else z)
    zh = y @ w.astype(np.float64) + 0.125
    want = nx.sigmoid(zh) if hact == rb.RB_ACT_SIGMOID else zh
    for i, rr in enumerate(sel):
        if out_idx[rr] >= 0:
            assert abs(g[out_idx[rr]] - want[i]) <= 2e-2 * max(abs(want[i]), 1e-2), (rr, g[out_idx[rr]], want[i])


def test_gemm_head_rejects_bad_arguments():
    st = _stream()
    X = torch.zeros((128, 128), dtype=torch.int16, device=DEV)
    W = torch.zeros((256, 128), dtype=torch.int16, device=DEV)
    w = torch.zeros(264, dtype=torch.int16, device=DEV)
    b = torch.zeros(256, device=DEV)
    out = torch.zeros(128, device=DEV)
    rows = _rows_dev(np.zeros(128), np.zeros(128), np.arange(128))
    lib = rb.lib()

    def call(K=128, ldx=128, wp=None, act=rb.RB_ACT_RELU, hact=rb.RB_ACT_SIGMOID):
        return lib.rb_k_gemm_head(st, rb.dptr(X), ldx, rb.dptr(W), 128, rb.dptr(b), 128, K, act, rb.dptr(rows),
                                  rb.dptr(w) if wp is None else wp, 0.0, hact, rb.dptr(out))
    assert call() == rb.RB_OK
    assert call(K=96) == rb.RB_EINVAL             # K not a multiple of 64
    assert call(ldx=64) == rb.RB_EINVAL           # ldx < K
    assert call(wp=rb.dptr(w) + 2) == rb.RB_EINVAL  # head weights not 16-byte aligned
    assert call(hact=rb.RB_ACT_RELU) == rb.RB_EINVAL
    torch.cuda.synchronize()


@pytest.mark.parametrize("S,T,D", [(50, 64, 256), (20, 512, 256), (30, 64, 100), (10, 128, 1000)])
def test_seqpool_matches_oracle(S, T, D):
    # float4 path (D % 4 == 0), scalar path, long sequences split over waves
    rng = np.random.default_rng(7)
    n_out = 2
    L = rng.integers(1, T + 1, size=S)
    L[:3] = [1, T, 2]
    H = rng.standard_normal((S * T, D)).astype(np.float32)
    Hn = H.copy()
    for s in range(S):
        Hn[s * T + L[s]:(s + 1) * T] = np.nan   # tokens past L must never be read
    Wh = (rng.standard_normal((n_out, D)) / 16).astype(np.float32)
    bh = rng.uniform(-0.5, 0.5, n_out).astype(np.float32)
    out_idx = np.arange(S) * n_out
    out_idx[5] = -1
    rows = _rows_dev(np.zeros(S), L, out_idx)
    out = torch.full((S * n_out,), -7.0, device=DEV)
    Hd, Whd, bhd = _dev(Hn), _dev(Wh), _dev(bh)
    rb.check(rb.lib().rb_k_seqpool(_stream(), rb.dptr(rows), S, T, 0, rb.dptr(Hd), D, D, rb.dptr(Whd),
                                   rb.dptr(bhd), n_out, rb.RB_ACT_SOFTMAX, rb.dptr(out)), "seqpool")
    # the same sequences packed: sequence s's tokens at rows [off_s, off_s + L_s)
    # of a [sum L, D] matrix, with NaN rows after it
    off = np.concatenate([[0], np.cumsum(L)[:-1]])
    Hp = np.concatenate([H[s * T:s * T + L[s]] for s in range(S)] + [np.full((7, D), np.nan, np.float32)])
    a = np.zeros(S, dtype=rb.K_ROW_DTYPE)
    a["src"], a["aux"], a["lens"], a["out"] = 0, L, off, out_idx
    rows_p = _dev(a.view(np.uint8))
    out_p = torch.full((S * n_out,), -7.0, device=DEV)
    Hpd = _dev(Hp)
    rb.check(rb.lib().rb_k_seqpool(_stream(), rb.dptr(rows_p), S, T, int(L.sum()), rb.dptr(Hpd), D, D, rb.dptr(Whd),
                                   rb.dptr(bhd), n_out, rb.RB_ACT_SOFTMAX, rb.dptr(out_p)), "seqpool packed")
    torch.cuda.synchronize()
    o = out.cpu().numpy().reshape(S, n_out)
    # same partition of each sequence, same order: bit-identical to the slot layout
    assert np.array_equal(out_p.cpu().numpy().reshape(S, n_out), o)
    for s in range(S):
        if out_idx[s] < 0:
            assert np.all(o[s] == -7.0)
            continue
        pooled = nx.round_f32(np.sum(H[s * T:s * T + L[s]].astype(np.float64), axis=0) / L[s])
        ref = nx.round_f32(nx.softmax(nx.round_f32(nx.dense(pooled[None], Wh, bh, "none"))))[0]
        assert np.max(np.abs(o[s] - ref)) <= 1e-5 * np.max(np.abs(ref)), s


@pytest.mark.parametrize("dt,M,N,K,d_out,gap", [
    ("bf16", 1000, 512, 256, 512, 0), ("bf16", 300, 4096, 512, 4096, 0), ("bf16", 4133, 256, 1728, 250, 3),
    ("bf16", 77, 128, 64, 7, 1), ("f32", 700, 64, 64, 16, 0), ("f32", 1234, 1024, 256, 1000, 2),
    ("f32", 33, 64, 32, 3, 5)])
def test_gemm_rows_out_bit_identical_to_gemm_and_split(dt, M, N, K, d_out, gap):
    # the last layer writing each real row's first d_out fp32 outputs through
    # the row map against the layer into Y followed by rb_k_split: the same
    # bits at every output position, nothing written for padding rows, past
    # d_out or between rows (gaps leave output offsets that are not multiples
    # of 4 floats: the element path)
    rng = np.random.default_rng(31)
    gaps = rng.integers(0, gap + 1, size=M)
    off = np.cumsum(np.concatenate([[0], (d_out + gaps)[:-1]]))
    out_idx = np.where(rng.random(M) < 0.85, off, -1)
    rows = _rows_dev(np.zeros(M), np.zeros(M), out_idx)
    n_out = int(off[-1]) + d_out + 8
    b = _dev(rng.uniform(-0.5, 0.5, N).astype(np.float32))
    st = _stream()
    Y = torch.empty((M, N), dtype=torch.float32, device=DEV)
    ref = torch.full((n_out,), -7.0, device=DEV)
    got = torch.full((n_out,), -7.0, device=DEV)
    lib = rb.lib()
    if dt == "bf16":
        Xd, _ = _bf16_dev(rng.standard_normal((M, K)))
        Wd, _ = _bf16_dev(rng.standard_normal((N, K)) / np.sqrt(K))
        rb.check(lib.rb_k_gemm_bf16(st, rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(b), rb.dptr(Y), N, M, N, K,
                                    rb.RB_ACT_NONE, 1), "gemm")
        rb.check(lib.rb_k_gemm_bf16_rows(st, rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(b), M, N, K, rb.RB_ACT_NONE,
                                         rb.dptr(rows), d_out, rb.dptr(got)), "gemm rows")
    else:
        Xd = _dev(rng.standard_normal((M, K)).astype(np.float32))
        Wd = _dev((rng.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32))
        rb.check(lib.rb_k_gemm_f32(st, rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(b), rb.dptr(Y), N, M, N, K,
                                   rb.RB_ACT_RELU, None, 0), "gemm")
        rb.check(lib.rb_k_gemm_f32_rows(st, rb.dptr(Xd), K, rb.dptr(Wd), K, rb.dptr(b), M, N, K, rb.RB_ACT_RELU,
                                        rb.dptr(rows), d_out, rb.dptr(got)), "gemm rows")
    rb.check(lib.rb_k_split(st, rb.dptr(rows), M, rb.dptr(Y), N, d_out, rb.dptr(ref)), "split")
    torch.cuda.synchronize()
    g, r = got.cpu().numpy(), ref.cpu().numpy()
    assert np.array_equal(g.view(np.uint32), r.view(np.uint32))
    assert np.sum(g != -7.0) <= int(np.sum(out_idx >= 0)) * d_out


def test_gemm_rows_out_rejects_bad_arguments():
    st = _stream()
    X = torch.zeros((64, 64), dtype=torch.int16, device=DEV)
    W = torch.zeros((128, 64), dtype=torch.int16, device=DEV)
    b = torch.zeros(128, device=DEV)
    out = torch.zeros(64 * 128, device=DEV)
    rows = _rows_dev(np.zeros(64), np.zeros(64), np.arange(64) * 128)
    lib = rb.lib()

    def call(N=128, d_out=128, rp=None):
        return lib.rb_k_gemm_bf16_rows(st, rb.dptr(X), 64, rb.dptr(W), 64, rb.dptr(b), 64, N, 64, rb.RB_ACT_NONE,
                                       rb.dptr(rows) if rp is None else rp, d_out, rb.dptr(out))
    assert call() == rb.RB_OK
    assert call(d_out=129) == rb.RB_EINVAL   # more outputs than the layer has
    assert call(d_out=0) == rb.RB_EINVAL
    assert call(rp=0) == rb.RB_EINVAL        # no row map
    assert call(N=96) == rb.RB_EINVAL        # N not a multiple of 128 (bf16)
    torch.cuda.synchronize()


@pytest.mark.parametrize("d_out,ldy", [(64, 64), (4096, 4096), (32, 64), (7, 8)])
def test_split_vector_and_scalar_paths(d_out, ldy):
    # output offsets mix multiples of 4 floats (16-byte path) and others
    rng = np.random.default_rng(8)
    R = 257
    gaps = rng.integers(0, 3, size=R)
    off = np.cumsum(np.concatenate([[0], (d_out + gaps)[:-1]]))
    out_idx = np.where(rng.random(R) < 0.9, off, -1)
    rows = _rows_dev(np.zeros(R), np.zeros(R), out_idx)
    Y = rng.standard_normal((R, ldy)).astype(np.float32)
    Yd = _dev(Y)
    out = torch.full((int(off[-1]) + d_out + 8,), -7.0, device=DEV)
    rb.check(rb.lib().rb_k_split(_stream(), rb.dptr(rows), R, rb.dptr(Yd), ldy, d_out, rb.dptr(out)), "split")
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    want = np.full_like(o, -7.0)
    for r in range(R):
        if out_idx[r] >= 0:
            want[out_idx[r]:out_idx[r] + d_out] = Y[r, :d_out]
    assert np.array_equal(o, want)
