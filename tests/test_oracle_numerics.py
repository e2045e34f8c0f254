"""Pins of the oracle's numerics against values fixed outside the oracle:
hand-worked examples, closed forms, exact rational brute force, and library
routines the oracle itself does not use (torch's bfloat16 conversion and
embedding_bag)."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import numerics as nx


# ---------------------------------------------------------------- bf16 rounding

def test_bf16_hand_cases():
    # ulp of bf16 at 1.0 is 2^-7
    cases = [
        (1.0, 1.0),
        (1 + 2 ** -8, 1.0),                      # tie -> even (1.0)
        (1 + 3 * 2 ** -8, 1 + 2 ** -6),          # tie -> even (fraction ...10)
        (1 + 2 ** -8 + 2 ** -30, 1 + 2 ** -7),   # just above the tie: up (no double rounding)
        (-(1 + 2 ** -8 + 2 ** -30), -(1 + 2 ** -7)),
        (0.0, 0.0),
        (2 ** -133, 2 ** -133),                  # smallest subnormal
        (2 ** -134, 0.0),                        # half the smallest subnormal: tie -> 0 (even)
        (3 * 2 ** -134, 2 ** -132),              # tie between 1 and 2 quanta -> 2 (even)
        (float.fromhex("0x1.fep127"), float.fromhex("0x1.fep127")),
        (float.fromhex("0x1.ffp127"), math.inf),   # max + half ulp (tie) -> inf (even)
        (float.fromhex("0x1.fefp127"), float.fromhex("0x1.fep127")),  # just below the tie
        (-math.inf, -math.inf),
    ]
    x = np.array([c[0] for c in cases])
    want = np.array([c[1] for c in cases])
    got = nx.round_bf16(x)
    assert np.array_equal(got, want), list(zip(x, got, want))
    assert np.isnan(nx.round_bf16(np.array([np.nan]))[0])
    assert math.copysign(1.0, nx.round_bf16(np.array([-0.0]))[0]) == -1.0


def test_bf16_matches_torch_on_fp32_values():
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 2 ** 32, size=200_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    ours = nx.round_bf16(x)
    theirs = torch.from_numpy(x.copy()).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, theirs)


def test_f32_rounding_is_binary32():
    x = np.array([1 + 2 ** -24, 1 + 3 * 2 ** -24, 0.1])
    got = nx.round_f32(x)
    assert got[0] == 1.0 and got[1] == 1 + 2 ** -22 and got[2] == float(np.float32(0.1))


# ---------------------------------------------------------------- dense layer

def test_dense_hand_worked(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "mlp_tiny.json")))
    x = np.array([g["x"]], dtype=np.float64)
    h = nx.dense(x, np.array(g["W1"]), np.array(g["b1"]), g["act1"])
    y = nx.dense(h, np.array(g["W2"]), np.array(g["b2"]), g["act2"])
    assert y.tolist() == [g["y"]]


def test_dense_zero_weights_give_act_of_bias():
    b = np.array([-1.5, 0.0, 2.25])
    h = np.random.default_rng(0).standard_normal((5, 4))
    assert np.array_equal(nx.dense(h, np.zeros((3, 4)), b, "relu"), np.tile([0.0, 0.0, 2.25], (5, 1)))
    assert np.array_equal(nx.dense(h, np.zeros((3, 4)), b, "none"), np.tile(b, (5, 1)))


def test_dense_permutation_weights_select_inputs():
    # W[j, perm[j]] = 1: output j is input perm[j]; a transposed W would give perm^-1
    n = 7
    perm = np.array([3, 0, 6, 1, 5, 2, 4])
    W = np.zeros((n, n))
    W[np.arange(n), perm] = 1.0
    h = np.random.default_rng(1).standard_normal((3, n))
    assert np.array_equal(nx.dense(h, W, np.zeros(n), "none"), h[:, perm])


def test_dense_exact_rational_bruteforce():
    # dyadic inputs: fp64 accumulation is exact, so it must equal exact rationals
    rng = np.random.default_rng(2)
    for _ in range(20):
        K, N, R = rng.integers(1, 9, size=3)
        h = rng.integers(-16, 17, size=(R, K)) / 8.0
        W = rng.integers(-16, 17, size=(N, K)) / 4.0
        b = rng.integers(-16, 17, size=N) / 2.0
        got = nx.dense(h, W, b, "relu")
        for r in range(R):
            for j in range(N):
                z = sum(Fraction(W[j, k]) * Fraction(h[r, k]) for k in range(K)) + Fraction(b[j])
                assert got[r, j] == float(max(z, Fraction(0)))


def test_sigmoid_and_softmax_closed_forms():
    assert nx.sigmoid(np.array([0.0]))[0] == 0.5
    z = np.linspace(-20, 20, 41)
    assert np.allclose(nx.sigmoid(z) + nx.sigmoid(-z), 1.0, rtol=0, atol=1e-15)
    assert np.all(np.diff(nx.sigmoid(z)) > 0)
    assert nx.sigmoid(np.array([math.log(3.0)]))[0] == pytest.approx(0.75, rel=1e-15)
    p = nx.softmax(np.array([[2.5, 2.5]]))
    assert p.tolist() == [[0.5, 0.5]]
    p = nx.softmax(np.array([[0.0, math.log(3.0)]]))
    assert np.allclose(p, [[0.25, 0.75]], rtol=1e-15)
    # shift invariance and huge logits (max subtraction keeps it finite)
    p1 = nx.softmax(np.array([[1000.0, 1000.0 + math.log(3.0)]]))
    assert np.allclose(p1, [[0.25, 0.75]], rtol=1e-12)


# ---------------------------------------------------------------- embedding bags

def test_embedding_bag_single_and_empty():
    T = np.random.default_rng(3).standard_normal((50, 8)).astype(np.float32)
    ids = np.array([7, 3, 49])
    out = nx.embedding_bag_sums(T, ids, np.array([1, 0, 1, 1]))
    assert np.array_equal(out[0], T[7].astype(np.float64))
    assert np.array_equal(out[1], np.zeros(8))
    assert np.array_equal(out[2], T[3].astype(np.float64))
    assert np.array_equal(out[3], T[49].astype(np.float64))


def test_embedding_bag_one_hot_histogram():
    # table row i = e_{i mod 8}: a bag's sum is the histogram of (id mod 8)
    T = np.zeros((40, 8), dtype=np.float32)
    T[np.arange(40), np.arange(40) % 8] = 1.0
    rng = np.random.default_rng(4)
    lens = rng.integers(0, 12, size=30)
    ids = rng.integers(0, 40, size=int(lens.sum()))
    out = nx.embedding_bag_sums(T, ids, lens)
    o = 0
    for i, L in enumerate(lens):
        hist = np.bincount(ids[o:o + L] % 8, minlength=8)
        assert np.array_equal(out[i], hist)
        o += L


def test_embedding_bag_matches_torch_embedding_bag():
    rng = np.random.default_rng(5)
    T = rng.standard_normal((200, 16))
    lens = rng.integers(1, 21, size=64)
    ids = rng.integers(0, 200, size=int(lens.sum()))
    ours = nx.embedding_bag_sums(T, ids, lens)
    offsets = np.concatenate([[0], np.cumsum(lens)[:-1]])
    theirs = torch.nn.functional.embedding_bag(torch.from_numpy(ids), torch.from_numpy(T),
                                               torch.from_numpy(offsets), mode="sum").numpy()
    assert np.allclose(ours, theirs, rtol=1e-13, atol=1e-13)
