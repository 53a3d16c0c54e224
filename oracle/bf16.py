"""bf16 <-> float64, written from the IEEE-754 definition (oracle; tests only).

bf16 is the upper half of an IEEE binary32: 1 sign bit, 8 exponent bits and 7
fraction bits, so it has binary32's exponent range (normal numbers from 2^-126,
subnormal spacing 2^-133) with 8 significant bits.  The paper trains in BF16
(Sec. 4.1); every bf16 value the library stores is produced by rounding to
nearest, ties to even.
"""
from __future__ import annotations

import numpy as np

BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127


def to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns, as float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):     # signalling-NaN patterns warn on widening
        return b.view(np.float32).astype(np.float64)


def from_f64(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16, ties to even; return the bits.

    Definition used: a finite |x| lies in a binade [2^E, 2^(E+1)); bf16 spaces
    its values there by q = 2^(max(E, -126) - 7) (the max covers subnormals).
    The result is q * rint(|x| / q), rint rounding half-way cases to the even
    integer.  A result above the largest finite bf16 becomes infinity.  NaN maps
    to the quiet NaN 0x7FC0 with the input's sign.
    """
    x = np.asarray(x, dtype=np.float64)
    sign = np.signbit(x)
    ax = np.abs(x)
    out = np.zeros(x.shape, dtype=np.float64)
    finite = np.isfinite(ax) & (ax > 0)
    if np.any(finite):
        a = ax[finite]
        _, e = np.frexp(a)          # a = m * 2^e, m in [0.5, 1)  ->  binade E = e - 1
        E = np.maximum(e - 1, -126)
        q = np.ldexp(1.0, E - 7)
        out[finite] = np.rint(a / q) * q
    out[np.isinf(ax)] = np.inf
    overflow = out > BF16_MAX
    out[overflow] = np.inf
    with np.errstate(over="ignore"):
        bits = (out.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    bits = np.where(sign, bits | np.uint16(0x8000), bits)
    nan = np.isnan(x)
    bits = np.where(nan, np.where(sign, np.uint16(0xFFC0), np.uint16(0x7FC0)), bits)
    return bits.astype(np.uint16)


def round_f64(x: np.ndarray) -> np.ndarray:
    """float64 -> nearest bf16 (ties to even) -> float64."""
    return to_f64(from_f64(x))
