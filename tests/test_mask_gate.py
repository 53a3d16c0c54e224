"""The mask comparison of the parity tests (tests/helpers.mask_gate) on
hand-made cases: it explains a disagreement only when the accumulation
range of h allows the GPU's choice, and it counts the relative window."""
import numpy as np

from tests.helpers import mask_gate, s_in_range


def _gate(gpu, ref, h, lo, hi):
    gpu, ref = np.array([gpu], dtype=bool), np.array([ref], dtype=bool)
    keys = np.maximum(np.array([h], dtype=np.float64), 0.0) ** 2
    return mask_gate(gpu, ref, keys, lambda rows, cols: (np.array([lo])[np.ix_(rows, cols)],
                                                        np.array([hi])[np.ix_(rows, cols)]))


def test_agreement():
    r = _gate([1, 1, 0, 0], [1, 1, 0, 0], [2.0, 1.0, 0.5, -1.0], [2.0, 1.0, 0.5, -1.0], [2.0, 1.0, 0.5, -1.0])
    assert r == {"groups": 1, "flips": 0, "outside_rel": 0, "unexplained": 0}


def test_flip_inside_the_range_is_explained():
    # h1 = 0.75 and h2 = 0.7539 (adjacent bf16), h1's range reaches 0.7539:
    # the GPU may rank h1 at 0.7539, tie with h2, and keep the lower index 1
    h = [1.0, 0.75, 0.75390625, -1.0]
    lo = [1.0, 0.75, 0.75390625, -1.0]
    hi = [1.0, 0.75390625, 0.75390625, -1.0]
    r = _gate([1, 1, 0, 0], [1, 0, 1, 0], h, lo, hi)
    assert r["flips"] == 1 and r["unexplained"] == 0
    assert r["outside_rel"] == 1          # 0.7539^2 / 0.75^2 - 1 = 1.04 % > 1e-2


def test_flip_outside_the_range_is_unexplained():
    h = [1.0, 0.75, 0.75390625, -1.0]
    r = _gate([1, 1, 0, 0], [1, 0, 1, 0], h, h, h)       # single-valued ranges
    assert r["unexplained"] == 1


def test_tie_breaks_to_the_lower_index():
    h = [1.0, 0.5, 0.5, 0.0]
    # tie between positions 1 and 2: keeping 2 over 1 cannot be explained
    assert _gate([1, 0, 1, 0], [1, 1, 0, 0], h, h, h)["unexplained"] == 1
    # but keeping 1 over 2 is the rule itself (no flip)
    assert _gate([1, 1, 0, 0], [1, 1, 0, 0], h, h, h)["flips"] == 0
    # negative h: relu keys tie at 0; the lower index wins
    hn = [1.0, -0.5, -0.25, -0.125]
    assert _gate([1, 1, 0, 0], [1, 1, 0, 0], hn, hn, hn)["flips"] == 0
    assert _gate([1, 0, 1, 0], [1, 1, 0, 0], hn, hn, hn)["unexplained"] == 1


def test_every_kept_dropped_pair_is_checked():
    # the GPU keeps the two smallest: no h in these ranges allows it
    h = [3.0, 2.0, 1.0, 0.5]
    assert _gate([0, 0, 1, 1], [1, 1, 0, 0], h, h, h)["unexplained"] == 1


def test_s_in_range():
    assert s_in_range(np.array([1.0, 2.0]), np.array([1.0, 1.5]), np.array([1.0, 2.0]))
    assert not s_in_range(np.array([1.0, 2.5]), np.array([1.0, 1.5]), np.array([1.0, 2.0]))
