"""Pins of oracle.bf16 (bf16 round-to-nearest-even from float64).

The oracle's rounding is checked against two things it does not share code
with: torch's float32 -> bfloat16 conversion (round to nearest even), and the
defining property of the result (it is a nearest bf16 value, and on a tie its
last bit is 0), checked through the bf16 neighbours obtained by stepping the
bit pattern.
"""
import numpy as np
import pytest
import torch

from oracle import bf16


def _torch_bf16_bits(f32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(f32.astype(np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_roundtrip_all_bf16_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    v = bf16.to_f64(bits)
    back = bf16.from_f64(v)
    nan = np.isnan(v)
    assert np.array_equal(back[~nan], bits[~nan])
    assert np.all((back[nan] & 0x7FFF) == 0x7FC0)


@pytest.mark.parametrize("lows", [[0x0000, 0x0001, 0x3FFF, 0x7FFF, 0x8000, 0x8001, 0xC000, 0xFFFF]])
def test_against_torch_every_upper_half(lows):
    hi = np.arange(1 << 16, dtype=np.uint32)
    for lo in lows:
        u = (hi << 16) | np.uint32(lo)
        f = u.view(np.float32)
        with np.errstate(invalid="ignore"):
            ours = bf16.from_f64(f.astype(np.float64))
        ref = _torch_bf16_bits(f)
        nan = np.isnan(f)
        assert np.array_equal(ours[~nan], ref[~nan]), hex(lo)
        assert np.all((ours[nan] & 0x7FFF) == 0x7FC0)


def test_against_torch_random_f32():
    g = np.random.default_rng(7)
    u = g.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    f = u.view(np.float32)
    with np.errstate(invalid="ignore"):      # signalling-NaN payloads warn on widening
        ours = bf16.from_f64(f.astype(np.float64))
    ref = _torch_bf16_bits(f)
    nan = np.isnan(f)
    assert np.array_equal(ours[~nan], ref[~nan])


def _neighbours_ok(x: np.ndarray):
    b = bf16.from_f64(x)
    v = bf16.to_f64(b)
    fin = np.isfinite(v) & (np.abs(v) < bf16.BF16_MAX)
    x, b, v = x[fin], b[fin], v[fin]
    # neighbours by stepping the magnitude bits (works across binades)
    mag = b & np.uint16(0x7FFF)
    sgn = b & np.uint16(0x8000)
    up = bf16.to_f64(sgn | (mag + np.uint16(1)))
    dn_mag = np.where(mag > 0, mag - np.uint16(1), mag)
    dn = bf16.to_f64(sgn | dn_mag)
    err = np.abs(x - v)
    assert np.all(err <= np.abs(x - up))
    assert np.all(err <= np.abs(x - dn))
    # other side of zero: -v's neighbour toward zero is covered by dn; a tie
    # must land on an even pattern
    tie = (err == np.abs(x - up)) | ((err == np.abs(x - dn)) & (mag > 0))
    assert np.all((b[tie] & 1) == 0)


def test_nearest_even_property_f64():
    g = np.random.default_rng(11)
    # float64 values with more precision than float32, all binades incl. subnormal bf16
    e = g.integers(-140, 128, size=200000)
    m = g.random(200000) + 1.0
    x = np.ldexp(m, e) * np.where(g.random(200000) < 0.5, -1.0, 1.0)
    _neighbours_ok(x)
    # exact midpoints between consecutive bf16 values
    bits = g.integers(0, 0x7F7F, size=100000).astype(np.uint16)
    lo = bf16.to_f64(bits)
    hi = bf16.to_f64(bits + np.uint16(1))
    mid = (lo + hi) / 2.0
    _neighbours_ok(mid)
    r = bf16.from_f64(mid)
    assert np.all((r & 1) == 0)


def test_special_values():
    x = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, bf16.BF16_MAX, 2.0 ** 128, -2.0 ** 128,
                  2.0 ** -133, 2.0 ** -134, 1.5 * 2.0 ** -134, 3.0 * 2.0 ** -135])
    b = bf16.from_f64(x)
    assert b[0] == 0x0000 and b[1] == 0x8000
    assert b[2] == 0x7F80 and b[3] == 0xFF80
    assert (b[4] & 0x7FFF) == 0x7FC0
    assert b[5] == 0x7F7F
    assert b[6] == 0x7F80 and b[7] == 0xFF80
    assert b[8] == 0x0001           # smallest subnormal
    assert b[9] == 0x0000           # half of it: tie -> even (zero)
    assert b[10] == 0x0001          # 0.75 of it -> 1
    assert b[11] == 0x0001          # 0.75 of smallest subnormal again
