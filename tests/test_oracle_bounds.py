"""Pins of oracle.bounds: the range of bf16 P and h that any binary32-
accumulating implementation of the up projection can produce.

* Simulated implementations (binary32 accumulation in random orders, rounding
  to nearest or toward zero, and blocked sums) always land inside the range.
* An implementation whose stored P rounds to either end of its own range
  (the case the dev_P term exists for) still lands inside the h range.
* Exact inputs (small integers times powers of two) give a single value,
  the oracle's own, wherever h is not 0; the oracle's h is always inside;
  lo <= hi.
"""
import numpy as np

from oracle import bf16 as obf
from oracle import bounds as obd
from oracle import ffn as offn
from synthetic import ffn_inputs, uniform_int_bf16


def _f32_sum(terms: np.ndarray, order: np.ndarray, toward_zero: bool) -> np.ndarray:
    """Sequential binary32 sum over the last axis of `terms` (float64 values
    exact in binary32) in the given order, rounding each addition to nearest
    or toward zero."""
    acc = np.zeros(terms.shape[:-1], dtype=np.float32)
    for k in order:
        s64 = acc.astype(np.float64) + terms[..., k]
        s32 = s64.astype(np.float32)
        if toward_zero:
            over = np.abs(s32.astype(np.float64)) > np.abs(s64)
            s32 = np.where(over, np.nextafter(s32, np.float32(0)), s32)
        acc = s32
    return acc.astype(np.float64)


def _f32_blocked(terms: np.ndarray, block: int) -> np.ndarray:
    """Blocks of `block` consecutive terms summed exactly (float64; at most
    16 bf16 products, so exact), each block added to a binary32 accumulator
    rounded to nearest: the shape of a matrix-core accumulation."""
    acc = np.zeros(terms.shape[:-1], dtype=np.float32)
    for k0 in range(0, terms.shape[-1], block):
        acc = (acc.astype(np.float64) + terms[..., k0:k0 + block].sum(axis=-1)).astype(np.float32)
    return acc.astype(np.float64)


def _simulate(a, x_rows, order_p, order_h, toward_zero, block=0):
    """bf16 P and h of one simulated implementation for the rows x_rows."""
    x, U, V = a["x"][x_rows], a["U_up"], a["V_up"]
    tp = x[:, :, None] * U[None, :, :]                      # [t, d, r]
    tp = np.moveaxis(tp, 1, 2)                              # [t, r, d]
    Pf = _f32_blocked(tp, block) if block else _f32_sum(tp, order_p, toward_zero)
    Pb = obf.round_f64(Pf)
    th = np.moveaxis(Pb[:, :, None] * V[None, :, :], 1, 2)  # [t, F, r]
    Hf = _f32_blocked(th, block) if block else _f32_sum(th, order_h, toward_zero)
    return Pb, obf.round_f64(Hf)


def test_simulated_accumulations_stay_inside():
    bits = ffn_inputs(24, 256, 64, 128, seed_base=91)
    a = offn.from_bits(bits)
    rows = np.arange(24)
    Pb, Plo, Phi = obd.stored_p_range(a["x"], a["U_up"])
    lo, hi = obd.h_range(a["x"], a["U_up"], a["V_up"])
    g = np.random.default_rng(4)
    cases = [(g.permutation(256), g.permutation(128), tz, 0) for tz in (False, True, False)]
    cases += [(None, None, False, 16)]
    for op, oh, tz, blk in cases:
        P, h = _simulate(a, rows, op, oh, tz, blk)
        assert np.all((Plo <= P) & (P <= Phi))
        assert np.all((lo <= h) & (h <= hi))


def test_stored_p_at_either_end_stays_inside():
    """P placed near bf16 rounding boundaries, so that many elements have two
    possible stored values; every element of P taken at a random end of its
    range, H accumulated from it in binary32: h stays inside."""
    g = np.random.default_rng(8)
    T, d, r, F = 32, 64, 96, 48
    # x U_up = k + 1/256 (+ tiny): just above a bf16 midpoint for k in [128, 256)
    x = np.zeros((T, d))
    x[:, 0] = g.integers(128, 256, T)
    x[:, 1] = 1.0
    U = np.zeros((d, r))
    U[0] = 1.0
    U[1] = 0.5                                       # P = k + 0.5: the midpoint between k and k + 1
    U[2:6] = g.choice([-1.0, 1.0], (4, r)) * 2.0 ** -20
    x[:, 2:6] = g.choice([-1.0, 1.0], (T, 4))
    V = obf.round_f64(g.standard_normal((r, F)) / np.sqrt(r))
    Pb, Plo, Phi = obd.stored_p_range(x, U)
    assert np.mean(Phi > Plo) > 0.5                 # the construction puts most of P on a boundary
    lo, hi = obd.h_range(x, U, V)
    for trial in range(3):
        pick = g.random(Pb.shape) < 0.5
        P = np.where(pick, Plo, Phi)
        th = np.moveaxis(P[:, :, None] * V[None, :, :], 1, 2)
        h = obf.round_f64(_f32_sum(th, g.permutation(r), trial == 2))
        assert np.all((lo <= h) & (h <= hi)), trial


def test_exact_inputs_give_a_single_value():
    T, d, F, r = 40, 64, 96, 40
    bits = {"x": uniform_int_bf16((T, d), -1, 1, 1), "U_up": uniform_int_bf16((d, r), -1, 1, 2),
            "V_up": uniform_int_bf16((r, F), -1, 1, 3, -2)}
    a = offn.from_bits(bits)
    lo, hi = obd.h_range(a["x"], a["U_up"], a["V_up"])
    Pb = obf.round_f64(a["x"] @ a["U_up"])
    h = obf.round_f64(Pb @ a["V_up"])
    # a single value wherever h != 0 (a zero sum has bf16 neighbours closer
    # than any accumulation bound, so its range straddles 0)
    nz = h != 0
    assert nz.mean() > 0.8
    np.testing.assert_array_equal(lo[nz], h[nz])
    np.testing.assert_array_equal(hi[nz], h[nz])
    assert np.all((lo[~nz] <= 0) & (hi[~nz] >= 0))


def test_oracle_h_inside_and_rows_cols_subsets():
    bits = ffn_inputs(50, 128, 200, 64, seed_base=12)
    a = offn.from_bits(bits)
    f = offn.forward(a["x"], a["U_up"], a["V_up"], a["U_down"], a["V_down"])
    lo, hi = obd.h_range(a["x"], a["U_up"], a["V_up"])
    assert np.all(lo <= hi)
    assert np.all((lo <= f["H"]) & (f["H"] <= hi))
    # the range holds more than one bf16 value only near rounding boundaries
    assert np.mean(lo < hi) < 0.8
    rows, cols = np.array([3, 7, 49]), np.array([0, 5, 199])
    slo, shi = obd.h_range(a["x"], a["U_up"], a["V_up"], rows, cols)
    np.testing.assert_array_equal(slo, lo[np.ix_(rows, cols)])
    np.testing.assert_array_equal(shi, hi[np.ix_(rows, cols)])


def test_exact_p_inputs_fix_p():
    """exact_p_inputs draw x and U_up so that P = x U_up is exact in binary32:
    the stored P has a single possible value, and h's range is narrower than
    for the unquantised inputs of the same shape."""
    from synthetic import exact_p_inputs
    for T, d, F, r in [(16, 2048, 64, 512), (16, 128, 64, 256)]:
        q = offn.from_bits(exact_p_inputs(T, d, F, r, seed_base=5))
        assert np.all(obd.exact_product(q["x"], q["U_up"]))
        Pb, Plo, Phi = obd.stored_p_range(q["x"], q["U_up"])
        np.testing.assert_array_equal(Plo, Phi)
        g = offn.from_bits(ffn_inputs(T, d, F, r, seed_base=5))
        wq = np.mean(np.subtract(*obd.h_range(q["x"], q["U_up"], q["V_up"])[::-1]))
        wg = np.mean(np.subtract(*obd.h_range(g["x"], g["U_up"], g["V_up"])[::-1]))
        assert wq < wg
        assert abs(q["x"].std() - 1) < 0.05 and abs(q["U_up"].std() * np.sqrt(d) - 1) < 0.1


def test_exact_product_detects_rounding():
    """exact_product: integers below 2^24 in total are exact; one more unit
    (2^24 + 1 is not a binary32 value) is not; a finer grid lowers the limit."""
    A = np.array([[2.0 ** 23, 2.0 ** 23 - 1.0]])
    B = np.array([[1.0], [1.0]])
    assert obd.exact_product(A, B)[0, 0]
    assert not obd.exact_product(np.array([[2.0 ** 23, 2.0 ** 23 + 1.0]]), B)[0, 0]
    assert not obd.exact_product(np.array([[2.0 ** 23, 0.5]]), B)[0, 0]
    assert obd.exact_product(np.array([[2.0 ** 22, 0.5]]), B)[0, 0]


def test_gamma():
    assert obd.gamma(512, 2.0 ** -23) == 512 * 2.0 ** -23 / (1 - 512 * 2.0 ** -23)
    import pytest
    with pytest.raises(ValueError):
        obd.gamma(2 ** 23, 2.0 ** -23)
