"""Oracle numerics: the per-row arithmetic of the served models, in fp64.

Test infrastructure only: nothing on the product path imports this module.

Storage roundings are part of the model definition. Accumulation is fp64, so
the oracle is the exact result up to one final rounding per stored value:

  fp32 models  every layer output is rounded to fp32;
  bf16 models  weights and embedding tables are stored bf16 (round to nearest
               even from the fp32 draw), every layer input is rounded to bf16,
               biases stay fp32, the activation is applied before rounding,
               and the last layer's output is rounded to fp32.

The paper (section 2.2.1) treats the model as a black box that is run once per
merged request; these functions define what that black box computes for one
row, so that "batched result == per-request result" can be checked.
"""
from __future__ import annotations

import numpy as np

BF16_MAX = float.fromhex("0x1.fep127")      # largest finite bfloat16
_BF16_MIN_EXP = -133                        # quantum of bfloat16 subnormals: 2^-133


def round_bf16(x) -> np.ndarray:
    """Round real values (fp32 or fp64) to the nearest bfloat16, ties to even.

    bfloat16 is binary32 with 8 significant bits: exponent range of fp32,
    subnormal quantum 2^-133. Returned as fp64 values that are exactly
    bfloat16-representable. NaN stays NaN; overflow goes to +/-inf (a value
    at or beyond max + half an ulp rounds to infinity under ties-to-even,
    because the tie candidate 2^128 has an even significand).
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    fin = np.isfinite(x)
    out[~fin] = x[~fin]
    xf = x[fin]
    _, e = np.frexp(xf)                    # xf = m * 2^e, 0.5 <= |m| < 1
    q = np.maximum(e - 8, _BF16_MIN_EXP)   # quantum: 8 significant bits
    y = np.rint(np.ldexp(xf, -q))          # rint = round half to even
    y = np.ldexp(y, q)
    y = np.where(np.abs(y) > BF16_MAX, np.copysign(np.inf, xf), y)
    out[fin] = y
    return out


def round_f32(x) -> np.ndarray:
    """Round to the nearest binary32 (ties to even), returned as fp64 values."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def relu(z: np.ndarray) -> np.ndarray:
    return np.maximum(z, 0.0)


def sigmoid(z: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-z))


def softmax(z: np.ndarray) -> np.ndarray:
    """Softmax over the last axis with the row maximum subtracted first."""
    m = np.max(z, axis=-1, keepdims=True)
    e = np.exp(z - m)
    return e / np.sum(e, axis=-1, keepdims=True)


ACTS = {"none": lambda z: z, "relu": relu, "sigmoid": sigmoid, "softmax": softmax}


def dense(h: np.ndarray, W: np.ndarray, b: np.ndarray, act: str) -> np.ndarray:
    """One dense layer on rows of h: act(h @ W^T + b), accumulated in fp64.

    h [rows, K], W [N, K] (output-major, K contiguous), b [N]; result fp64
    [rows, N] before any storage rounding.
    """
    z = np.asarray(h, np.float64) @ np.asarray(W, np.float64).T + np.asarray(b, np.float64)
    return ACTS[act](z)


def embedding_bag_sums(table: np.ndarray, ids: np.ndarray, lens: np.ndarray) -> np.ndarray:
    """Sum-pool consecutive bags of ids: bag i is the next lens[i] ids.

    Row i of the result is the fp64 sum, in bag order, of table[id] over bag
    i's ids; an empty bag sums to zeros. table [rows, dim]; ids [sum(lens)];
    result [len(lens), dim].
    """
    lens = np.asarray(lens, dtype=np.int64)
    out = np.zeros((lens.shape[0], table.shape[1]), dtype=np.float64)
    if ids.size == 0:
        return out
    rows = np.asarray(table)[np.asarray(ids, dtype=np.int64)].astype(np.float64)
    starts = np.zeros(lens.shape[0], dtype=np.int64)
    np.cumsum(lens[:-1], out=starts[1:])
    nz = lens > 0
    # add.reduceat sums each segment left to right; empty segments are masked
    out[nz] = np.add.reduceat(rows, starts[nz], axis=0)
    return out
