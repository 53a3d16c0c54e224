"""Pins of oracle.ffn.fullrank_forward, the full-rank ReLU^2 FFN that Table 3
(Sec. 4.2.3) compares ELAS against.

* Brute force: explicit loops over tokens, features and outputs on tiny shapes.
* Factorisation: with W_up = (U_up V_up)^T and W_down = (U_down V_down)^T
  (Eq. 1, W = A B with U = B^T, V = A^T) the block
  equals the low-rank block with dense activations (the low-rank oracle is
  itself pinned against torch autograd).
* Closed forms: all pre-activations <= 0 gives exact zeros; scaling x by 2
  scales Y by exactly 4 (ReLU^2 is 2-homogeneous and power-of-two scaling
  commutes with bf16 rounding).
"""
import numpy as np

from oracle import bf16, ffn


def _rand(shape, g, scale=1.0):
    return g.standard_normal(shape) * scale


def test_brute_force_loops():
    g = np.random.default_rng(11)
    T, d, F = 3, 4, 8
    x, Wu, Wd = _rand((T, d), g), _rand((F, d), g, 0.5), _rand((d, F), g, 0.3)
    f = ffn.fullrank_forward(x, Wu, Wd, bf16io=False)
    want = np.zeros((T, d))
    for t in range(T):
        for j in range(d):
            acc = 0.0
            for k in range(F):
                h = sum(x[t, i] * Wu[k, i] for i in range(d))
                acc += (h if h > 0 else 0.0) ** 2 * Wd[j, k]
            want[t, j] = acc
    np.testing.assert_allclose(f["Y"], want, rtol=1e-12, atol=1e-14)
    assert (f["S"] >= 0).all() and ((f["S"] > 0) == (f["H"] > 0)).all()


def test_factorised_weights_equal_dense_low_rank_block():
    g = np.random.default_rng(12)
    T, d, F, r = 7, 16, 24, 8
    x = _rand((T, d), g)
    U_up, V_up = _rand((d, r), g, d ** -0.5), _rand((r, F), g, r ** -0.5)
    U_down, V_down = _rand((F, r), g, F ** -0.5), _rand((r, d), g, r ** -0.5)
    full = ffn.fullrank_forward(x, (U_up @ V_up).T, (U_down @ V_down).T, bf16io=False)
    low = ffn.forward(x, U_up, V_up, U_down, V_down, bf16io=False, sparse=False)
    np.testing.assert_allclose(full["S"], low["s"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(full["Y"], low["Y"], rtol=1e-10, atol=1e-12)


def test_nonpositive_preactivations_give_zero():
    g = np.random.default_rng(13)
    T, d, F = 6, 8, 16
    x = np.abs(_rand((T, d), g))
    Wu = -np.abs(_rand((F, d), g))
    Wd = _rand((d, F), g)
    for io in (False, True):
        f = ffn.fullrank_forward(x, Wu, Wd, bf16io=io)
        assert not f["S"].any() and not f["Y"].any()


def test_scaling_is_quadratic_and_rounding_points():
    g = np.random.default_rng(14)
    T, d, F = 5, 16, 32
    x = bf16.round_f64(_rand((T, d), g))
    Wu = bf16.round_f64(_rand((F, d), g, d ** -0.5))
    Wd = bf16.round_f64(_rand((d, F), g, F ** -0.5))
    for io in (False, True):
        a = ffn.fullrank_forward(x, Wu, Wd, bf16io=io)
        b = ffn.fullrank_forward(2.0 * x, Wu, Wd, bf16io=io)
        np.testing.assert_array_equal(b["Y"], 4.0 * a["Y"])
    f = ffn.fullrank_forward(x, Wu, Wd, bf16io=True)
    for k in ("H", "S", "Y"):
        assert np.array_equal(bf16.round_f64(f[k]), f[k]), k
