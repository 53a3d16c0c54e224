"""Pins of oracle.sparsify (Eq. 2, Algorithm 1, Eq. 3 and the compressed layout).

* Brute force: every group is checked against an enumeration of the 6
  possible keep patterns (a pattern is valid when no dropped magnitude exceeds
  a kept one; among valid patterns the one with the lexicographically smallest
  sorted index pair is the stable top-2).  Only comparisons are used.
* Invariants of a 2:4 result, a hand-worked example, and the storage ratio of
  Table 2.
"""
import itertools
import os

import numpy as np
import pytest

from oracle import bf16, sparsify

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
PATTERNS = list(itertools.combinations(range(4), 2))   # (0,1),(0,2),...,(2,3): lexicographic


def brute_keep(keys):
    """Keep-pair of one group by enumeration of the 6 patterns (pure Python)."""
    for pat in PATTERNS:
        kept = [keys[i] for i in pat]
        dropped = [keys[i] for i in range(4) if i not in pat]
        if min(kept) >= max(dropped):
            return pat
    raise AssertionError("no valid pattern")


def _check_against_brute(z, keys):
    mask = sparsify.top2_mask(z)
    M, N = z.shape
    for i in range(M):
        for j in range(N // 4):
            pat = brute_keep([keys[i, 4 * j + k] for k in range(4)])
            want = np.zeros(4, dtype=bool)
            want[list(pat)] = True
            assert np.array_equal(mask[i, 4 * j:4 * j + 4], want), (keys[i, 4 * j:4 * j + 4], pat)


def test_brute_force_relu2_all_625_tuples():
    vals = [-2.0, -1.0, 0.0, 1.0, 2.0]
    tuples = np.array(list(itertools.product(vals, repeat=4)))     # 625 x 4
    h = tuples.reshape(1, -1)
    s = sparsify.relu2(h)
    _check_against_brute(s, s)


def test_brute_force_raw_all_256_tuples_signed():
    vals = [0.0, 1.0, 2.0, 3.0]
    tuples = np.array(list(itertools.product(vals, repeat=4)))
    signs = np.where(np.arange(tuples.size).reshape(tuples.shape) % 3 == 0, -1.0, 1.0)
    z = (tuples * signs).reshape(1, -1)
    _check_against_brute(z, np.abs(z))


def test_brute_force_random_rows():
    g = np.random.default_rng(3)
    z = np.round(g.standard_normal((16, 64)) * 2) / 2       # many ties
    _check_against_brute(z, np.abs(z))
    s = sparsify.relu2(g.standard_normal((16, 64)))
    _check_against_brute(s, s)


def test_invariants_random():
    g = np.random.default_rng(5)
    h = g.standard_normal((257, 1376)) + g.choice([-1.0, 0.0], size=(257, 1376))
    s = sparsify.relu2(h)
    mask = sparsify.top2_mask(s)
    km = mask.reshape(257, -1, 4)
    ks = s.reshape(257, -1, 4)
    assert np.all(km.sum(-1) == 2)
    kept_min = np.where(km, ks, np.inf).min(-1)
    drop_max = np.where(~km, ks, -np.inf).max(-1)
    assert np.all(kept_min >= drop_max)
    npos = (ks > 0).sum(-1)
    nz_kept = ((ks > 0) & km).sum(-1)
    assert np.array_equal(nz_kept, np.minimum(2, npos))
    S = sparsify.sparsify24(s)
    assert np.array_equal(S, np.where(mask, s, 0.0))
    vals, meta = sparsify.compress(S, mask)
    codes = np.concatenate([meta & 0xF, meta >> 4], axis=1)
    legal = {p[0] | (p[1] << 2) for p in PATTERNS}
    assert set(np.unique(codes).tolist()) <= legal
    dense, m2 = sparsify.decompress(vals, meta, 1376)
    assert np.array_equal(dense, S) and np.array_equal(m2, mask)


def _read_golden():
    rows = {}
    with open(os.path.join(GOLDEN, "sparsify_hand_example.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            k, *v = line.split()
            rows[k] = v
    return rows


def test_hand_example():
    g = _read_golden()
    h = np.array([float(v) for v in g["h"]])
    hb = bf16.from_f64(h).reshape(1, -1)
    for mode, key in ((sparsify.RELU2, "relu2"), (sparsify.RAW, "raw")):
        vals, meta = sparsify.sparsify24_bf16(hb, mode)
        want_vals = np.array([float(v) for v in g[key + "_vals"]])
        want_meta = np.array([int(v, 16) for v in g[key + "_meta"]], dtype=np.uint8)
        assert np.array_equal(bf16.to_f64(vals[0]), want_vals), key
        assert np.array_equal(meta[0], want_meta), key


def test_relu2_exact_and_monotone_on_every_bf16():
    """s = relu(h)^2 is exact in float64 for every finite bf16 h and strictly
    increasing over positive h, so ordering by s equals ordering by relu(h)."""
    bits = np.arange(0x0001, 0x7F80, dtype=np.uint32).astype(np.uint16)   # positive finite
    h = bf16.to_f64(bits)
    s = sparsify.relu2(h)
    assert np.all(np.diff(s) > 0)
    # exactness: the 8-bit significand squared fits in 16 bits, far below 53
    m, e = np.frexp(h)
    assert np.all(np.ldexp(m * m, 2 * e) == s)
    assert np.all(sparsify.relu2(-h) == 0) and sparsify.relu2(np.array([np.nan]))[0] == 0


def test_storage_ratio_matches_table2():
    """Kept bf16 values (half the entries) plus a 2-bit index per kept value,
    over dense bf16: (N/2*2 + N/8) / (2N) = 0.5625.  Table 2 gives
    ELAS/LORO = 0.560-0.563 at every batch size."""
    N = 5464
    vals_bytes = (N // 2) * 2
    meta_bytes = N // 8
    ratio = (vals_bytes + meta_bytes) / (2 * N)
    assert ratio == 0.5625
    rows = np.loadtxt(os.path.join(GOLDEN, "table2_activation_memory.txt"))
    paper = rows[:, 2] / rows[:, 1]
    assert np.all(np.abs(paper - ratio) < 0.005), paper
    # and the LORO column scales linearly with batch (dense activations)
    assert np.allclose(rows[:, 1] / rows[:, 0], rows[0, 1], rtol=0.01)


def test_shape_errors():
    with pytest.raises(ValueError):
        sparsify.top2_mask(np.zeros((2, 6)))
    with pytest.raises(ValueError):
        sparsify.compress(np.zeros((1, 4)), np.array([[True, True, False, False]]))
