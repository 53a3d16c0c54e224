"""Pins of oracle.ffn (the low-rank ReLU^2 2:4 FFN, forward and backward).

* torch autograd (float64, CPU) on the same block, built from
  torch.nn.functional.linear with the mask from the brute-force enumerator of
  test_oracle_sparsify, pins every output and gradient of the masked mode;
  a custom autograd function whose backward is the identity pins the
  straight-through mode of Eq. 4.
* Central finite differences of the full forward (the mask recomputed at every
  point) pin the masked gradients as the true derivative away from ties.
* Closed-form special cases: all h <= 0 gives zero output and zero weight
  gradients; at most 2 positives per group makes the block the dense low-rank
  ReLU^2 FFN and the two backward modes equal; T = 1.
"""
import numpy as np
import pytest
import torch

from oracle import bf16, ffn, sparsify
from tests.test_oracle_sparsify import brute_keep


def _rand(shape, g, scale=1.0):
    return g.standard_normal(shape) * scale


def _inputs(T, d, F, r, seed=0, shift=0.0):
    g = np.random.default_rng(seed)
    a = dict(x=_rand((T, d), g), U_up=_rand((d, r), g, d ** -0.5), V_up=_rand((r, F), g, r ** -0.5),
             U_down=_rand((F, r), g, F ** -0.5), V_down=_rand((r, d), g, r ** -0.5),
             dY=_rand((T, d), g))
    if shift:
        a["x"] = a["x"]  # keep
    return a


def _brute_mask(s):
    M, N = s.shape
    m = np.zeros_like(s, dtype=bool)
    for i in range(M):
        for j in range(N // 4):
            for k in brute_keep(list(s[i, 4 * j:4 * j + 4])):
                m[i, 4 * j + k] = True
    return m


class _STE(torch.autograd.Function):
    @staticmethod
    def forward(ctx, z, mask):
        return z * mask

    @staticmethod
    def backward(ctx, g):
        return g, None


def _torch_block(a, ste):
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=(k != "dY")) for k, v in a.items()}
    F = torch.nn.functional
    P = F.linear(t["x"], t["U_up"].T)
    H = F.linear(P, t["V_up"].T)
    s = torch.relu(H) ** 2
    mask = torch.tensor(_brute_mask(s.detach().numpy()), dtype=torch.float64)
    S = _STE.apply(s, mask) if ste else s * mask
    Z = F.linear(S, t["U_down"].T)
    Y = F.linear(Z, t["V_down"].T)
    (Y * t["dY"]).sum().backward()
    out = {"Y": Y.detach().numpy()}
    for k in ("x", "U_up", "V_up", "U_down", "V_down"):
        out["d" + k] = t[k].grad.numpy()
    return out


def _oracle(a, ste=False, bf16io=False, sparse=True):
    f = ffn.forward(a["x"], a["U_up"], a["V_up"], a["U_down"], a["V_down"], bf16io=bf16io, sparse=sparse)
    b = ffn.backward(a["dY"], a["x"], a["U_up"], a["V_up"], a["U_down"], a["V_down"], f,
                     bf16io=bf16io, ste=ste)
    return f, b


@pytest.mark.parametrize("ste", [False, True])
@pytest.mark.parametrize("shape", [(5, 16, 24, 4), (1, 8, 8, 8), (33, 24, 40, 8)])
def test_against_torch_autograd(shape, ste):
    a = _inputs(*shape, seed=sum(shape))
    f, b = _oracle(a, ste=ste)
    ref = _torch_block(a, ste)
    np.testing.assert_allclose(f["Y"], ref["Y"], rtol=1e-12, atol=1e-12)
    for k in ("dx", "dU_up", "dV_up", "dU_down", "dV_down"):
        np.testing.assert_allclose(b[k], ref[k], rtol=1e-11, atol=1e-12, err_msg=k)


def _loss(a):
    f = ffn.forward(a["x"], a["U_up"], a["V_up"], a["U_down"], a["V_down"], bf16io=False)
    return float((f["Y"] * a["dY"]).sum())


def test_finite_differences_masked_is_true_gradient():
    a = _inputs(3, 8, 8, 2, seed=42)
    f, b = _oracle(a)
    eps = 1e-6
    for name in ("x", "U_up", "V_up", "U_down", "V_down"):
        num = np.zeros_like(a[name])
        it = np.nditer(a[name], flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            ap = {k: v.copy() for k, v in a.items()}
            am = {k: v.copy() for k, v in a.items()}
            ap[name][idx] += eps
            am[name][idx] -= eps
            fp = ffn.forward(ap["x"], ap["U_up"], ap["V_up"], ap["U_down"], ap["V_down"], bf16io=False)
            fm = ffn.forward(am["x"], am["U_up"], am["V_up"], am["U_down"], am["V_down"], bf16io=False)
            assert np.array_equal(fp["mask"], f["mask"]) and np.array_equal(fm["mask"], f["mask"]), \
                "mask changed inside the difference step: pick another seed"
            num[idx] = (_loss(ap) - _loss(am)) / (2 * eps)
        np.testing.assert_allclose(b["d" + name], num, rtol=1e-6, atol=1e-8, err_msg=name)


def test_all_h_nonpositive_gives_zero():
    a = _inputs(7, 16, 16, 4, seed=1)
    a["V_up"] = -np.abs(a["V_up"])
    a["x"] = np.abs(a["x"])
    a["U_up"] = np.abs(a["U_up"])          # P >= 0, V_up <= 0  ->  H <= 0
    f, b = _oracle(a)
    assert np.all(f["H"] <= 0)
    assert np.all(f["Y"] == 0)
    for k in ("dx", "dU_up", "dV_up", "dU_down", "dV_down"):
        assert np.all(b[k] == 0), k
    assert np.any(b["dZ"] != 0)


def test_at_most_two_positives_equals_dense_and_ste():
    """If every group has <= 2 positive h, Algorithm 1 prunes only zeros: the
    block equals the dense low-rank ReLU^2 FFN (Eq. 2 without sparsify), and
    the masked and straight-through gradients agree (pruned slots have
    relu(h) = 0)."""
    T, d, F, r = 6, 8, 16, 4
    g = np.random.default_rng(9)
    # H = P V_up with P = x U_up; force H's sign pattern by choosing P = e_0
    a = _inputs(T, d, F, r, seed=9)
    a["U_up"] = np.zeros((d, r)); a["U_up"][0, 0] = 1.0
    a["x"][:, 0] = np.abs(a["x"][:, 0]) + 0.1                 # P[:,0] > 0, rest 0
    sign = np.tile([1.0, 1.0, -1.0, -1.0], F // 4)
    a["V_up"] = np.zeros((r, F)); a["V_up"][0] = sign * (np.abs(g.standard_normal(F)) + 0.1)
    fs, bs = _oracle(a)
    fd, bd = _oracle(a, sparse=False)
    _, bt = _oracle(a, ste=True)
    assert np.array_equal(fs["Y"], fd["Y"])
    for k in ("dx", "dU_up", "dV_up", "dU_down", "dV_down"):
        np.testing.assert_array_equal(bs[k], bd[k])
        np.testing.assert_array_equal(bs[k], bt[k])


def test_identity_up_factor_is_full_rank_ffn():
    """r = d and U_up = I: the block is W_down relu^2(W_up x) with W_up^T =
    V_up, sparsified (Eq. 2 + Eq. 3 on a full-rank up projection)."""
    T, d, F = 5, 8, 12
    a = _inputs(T, d, F, d, seed=4)
    a["U_up"] = np.eye(d)
    f, _ = _oracle(a)
    s = sparsify.relu2(a["x"] @ a["V_up"])
    want = (np.where(_brute_mask(s), s, 0) @ a["U_down"]) @ a["V_down"]
    np.testing.assert_allclose(f["Y"], want, rtol=1e-12, atol=1e-13)


def test_bf16io_rounds_stored_tensors():
    a = _inputs(9, 16, 24, 8, seed=2)
    f, b = _oracle(a, bf16io=True)
    for k in ("P", "H", "S", "Z", "Y"):
        assert np.array_equal(bf16.round_f64(f[k]), f[k]), k
    for k in ("dZ", "dH", "dP", "dx"):
        assert np.array_equal(bf16.round_f64(b[k]), b[k]), k
    f64, b64 = _oracle(a, bf16io=False)
    rel = np.linalg.norm(f["Y"] - f64["Y"]) / np.linalg.norm(f64["Y"])
    assert rel < 3e-2
