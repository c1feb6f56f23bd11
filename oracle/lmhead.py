"""LM-head logits and their row statistics, written from their definitions.

TEST INFRASTRUCTURE ONLY: imported by tests/ and the cpu_baseline leg of
bench.py, never by the library.

The verifier's inputs are the per-node distributions M_b(.|X^i) and
M_s(.|X^i) of the problem statement (Alg. 3, REQUIRE); each is
softmax(logits / T) of one row, where the row is an LM head's product of the
node's hidden state with the output embedding. These functions compute, in
float64:

* ``logits(hidden, weight)``: sum_k hidden[m][k] * weight[n][k] for bfloat16
  inputs (given as uint16 bit patterns, widened exactly): the exact product
  up to float64 rounding (numpy's matmul is the library primitive);
* ``row_stats(z, T)``: per row, the maximum and sum_n exp((z - max) / T), the
  two numbers that normalise softmax(z / T).
"""

from __future__ import annotations

import numpy as np

from .tv_oracle import to_f64


def logits(hidden, weight) -> np.ndarray:
    """hidden [M][K] and weight [N][K] (bf16 bits or floats) -> float64 [M][N]."""
    x = to_f64(hidden)
    w = to_f64(weight)
    return x @ w.T


def accumulation_bound(hidden, weight) -> np.ndarray:
    """Per entry, the sum over k of |hidden[m][k] * weight[n][k]|: any
    accumulation of the K products in float32 is within K * 2^-24 times this
    of the exact sum."""
    return np.abs(to_f64(hidden)) @ np.abs(to_f64(weight)).T


def row_stats(z, T: float):
    """(max, sum exp((z - max) / T)) of every row of z in float64, for the
    float32 temperature T. A row holding NaN or +inf gets a NaN or infinite
    sum; a row whose entries are all -inf gets max -inf and sum 0."""
    z = to_f64(z)
    T = float(np.float32(T))
    m = z.max(axis=-1)
    with np.errstate(invalid="ignore", over="ignore"):
        s = np.exp((z - m[..., None]) / T).sum(axis=-1)
    s = np.where(np.isneginf(m), 0.0, s)
    return m, s
