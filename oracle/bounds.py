"""Accumulation error bounds of the block's up projection (oracle; tests only).

The block forms P = x U_up and H = P V_up (Eq. 1 factors, Fig. 1 caption)
and ranks the ReLU^2 of h, H rounded to bf16, inside every group of 4
(Eq. 2, Algorithm 1).  An implementation that multiplies bf16 operands and
accumulates in binary32 (the products of two bf16 values are exact there:
8 + 8 significant bits) and rounds P and H to bf16 at the same points as
``ffn.forward(bf16io=True)`` reaches the exact sums only up to its
accumulation error.  Where an exact sum lies within that error of a bf16
rounding boundary the two can round to neighbouring bf16 values, and where
that moves a ranked key onto, or past, a competing one the 2:4 selection can
differ.  This module bounds the bf16 values any such implementation can
produce, from the arithmetic alone (no knowledge of its summation order).

Bound used (Higham, Accuracy and Stability of Numerical Algorithms, 2nd ed.,
Sec. 4.2, summation in any order): a sum of n terms computed by n - 1
floating-point additions with unit roundoff u satisfies

    |fl(sum) - sum| <= gamma_n * sum |terms|,   gamma_n = n u / (1 - n u)

(gamma_n over-covers gamma_{n-1}).  u = 2^-24 is binary32 with rounding to
nearest; ``ACC_UNIT`` = 2^-23 also covers an accumulator that rounds toward
zero, since matrix-core accumulation order and rounding are not specified.
The float64 sums computed here carry their own error, bounded the same way
with u = 2^-53 and added to the binary32 term.

A product is exact in binary32, whatever the order, when every term is a
multiple of 2^q and the sum of the terms' magnitudes is below 2^(24 + q):
every partial sum is then a multiple of 2^q below 2^(24 + q) in magnitude,
which binary32 represents.  Its error bound is then 0.

The two products chain: P's accumulated value lies within e_P of the exact
P (computed here in float64, the float64 error included; e_P = 0 where the
product is exact), so the bf16 P an implementation stores is one of
bf16(P - e_P) .. bf16(P + e_P) (rounding to nearest is monotone); let dev_P
be the largest distance of those from the oracle's bf16 P.  Then H
accumulated from that stored P lies within

    w = sum_k dev_P[k] |V_up[k]|  +  gamma_r sum_k (|P_b[k]| + dev_P[k]) |V_up[k]|

of H_b = P_b V_up, P_b being the oracle's bf16 P, and the bf16 h is one of
bf16(H_b - w) .. bf16(H_b + w).
"""
from __future__ import annotations

import numpy as np

from . import bf16
from .sparsify import relu2

ACC_UNIT = 2.0 ** -23      # binary32 accumulation, covering round-to-nearest and toward zero
F64_UNIT = 2.0 ** -53      # float64 rounding to nearest


def gamma(n: int, u: float) -> float:
    """gamma_n = n u / (1 - n u) (requires n u < 1)."""
    nu = n * u
    if nu >= 1.0:
        raise ValueError("n u must be below 1")
    return nu / (1.0 - nu)


def lowest_bit_log2(a: np.ndarray, axis: int) -> np.ndarray:
    """Largest q such that every nonzero entry along ``axis`` is a multiple
    of 2^q (float64 input; 1100 where all entries are zero)."""
    m, e = np.frexp(np.abs(a))                     # |a| = m 2^e, m in [0.5, 1)
    mi = (m * 2.0 ** 53).astype(np.int64)          # integer significand, |a| = mi 2^(e - 53)
    low = np.log2((mi & -mi).astype(np.float64), where=mi > 0, out=np.zeros(a.shape))
    q = np.where(mi > 0, e - 53 + low, 1100.0)
    return q.min(axis=axis)


def exact_product(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Boolean [rows of A, columns of B]: the entry of A B is exact in
    binary32 for every summation order (terms multiples of 2^q, their
    magnitudes summing below 2^(24 + q))."""
    q = lowest_bit_log2(A, 1)[:, None] + lowest_bit_log2(B, 0)[None, :]
    S = np.abs(A) @ np.abs(B)
    return S < np.ldexp(1.0, np.minimum(24 + q, 1000).astype(np.int64))


def stored_p_range(x: np.ndarray, U_up: np.ndarray, u: float = ACC_UNIT):
    """(P_b, P_lo, P_hi) for P = x U_up: the oracle's bf16 P and the smallest
    and largest bf16 value an implementation accumulating with unit roundoff
    u can store for each element (float64 arrays of exact bf16 values)."""
    d = x.shape[1]
    P = x @ U_up
    e = (gamma(d, u) + gamma(d, F64_UNIT)) * (np.abs(x) @ np.abs(U_up))
    e = np.where(exact_product(x, U_up), 0.0, e)
    return bf16.round_f64(P), bf16.round_f64(P - e), bf16.round_f64(P + e)


def h_range(x: np.ndarray, U_up: np.ndarray, V_up: np.ndarray, rows=None, cols=None,
            u: float = ACC_UNIT):
    """(h_lo, h_hi): the smallest and largest bf16 h = bf16(P V_up) that an
    implementation of the two accumulating products can produce, for the
    token rows ``rows`` and feature columns ``cols`` (index arrays or None
    for all).  float64 arrays of exact bf16 values, shape [rows, cols]."""
    xs = x if rows is None else x[rows]
    V = V_up if cols is None else V_up[:, cols]
    r = U_up.shape[1]
    Pb, Plo, Phi = stored_p_range(xs, U_up, u)
    dev = np.maximum(Phi - Pb, Pb - Plo)
    aV = np.abs(V)
    Hb = Pb @ V
    acc = (gamma(r, u) + gamma(r, F64_UNIT)) * ((np.abs(Pb) + dev) @ aV)
    fixed = ~np.any(dev > 0, axis=1)[:, None]      # rows whose stored P has one possible value
    acc = np.where(fixed & exact_product(Pb, V), 0.0, acc)
    w = dev @ aV + acc
    return bf16.round_f64(Hb - w), bf16.round_f64(Hb + w)


def s_range(h_lo: np.ndarray, h_hi: np.ndarray):
    """(s_lo, s_hi): bf16(relu(h)^2) at the two ends of an h range; s is
    monotone in h, so every possible stored dense activation lies between."""
    return bf16.round_f64(relu2(h_lo)), bf16.round_f64(relu2(h_hi))
