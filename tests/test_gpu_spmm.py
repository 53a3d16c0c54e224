"""elas_spmm_24 (2:4 sparse x dense on v_smfmac) against the oracle.

With small-integer operands every partial sum is exact in fp32 and float64,
so the single bf16 rounding of the result must agree bit for bit; with
Gaussian operands the result is compared within bf16 rounding."""
import numpy as np
import pytest
import torch

import paper_2605_03667_amd as elas
from oracle import bf16 as obf
from oracle import sparsify as osp
from synthetic import h_input, normal_bf16, uniform_int_bf16
from tests.helpers import dev_bf16, host_bits, pad_compressed, rel_fro

pytestmark = pytest.mark.gpu

SHAPES = [(1, 8, 8), (5, 40, 24), (64, 64, 8), (300, 1376, 128), (257, 5464, 136), (1000, 2048, 512),
          (513, 2736, 256), (129, 5464, 512)]


def _operands(M, K, N, seed, exact):
    if exact:
        h = uniform_int_bf16((M, K), -2, 2, seed)              # s in {0, 1, 4}
        b = uniform_int_bf16((K, N), -2, 2, seed + 1)
    else:
        h = h_input(M, K, seed)
        b = normal_bf16((K, N), 1.0 / np.sqrt(K), seed + 1)
    vals, meta = osp.sparsify24_bf16(h)
    dense, _ = osp.decompress(obf.to_f64(vals), meta, K)
    ref = dense @ obf.to_f64(b)
    return vals, meta, b, ref


def _gpu(vals, meta, b_kn, K, layout):
    pv, pm = pad_compressed(vals, meta, K)
    b = b_kn if layout == elas.ELAS_B_KN else np.ascontiguousarray(b_kn.T)
    c = elas.elas_spmm_24(dev_bf16(pv), torch.from_numpy(pm).to("cuda:0"), K, dev_bf16(b), layout)
    torch.cuda.synchronize()
    return host_bits(c)


@pytest.mark.parametrize("layout", [elas.ELAS_B_NK, elas.ELAS_B_KN])
@pytest.mark.parametrize("M,K,N", SHAPES)
def test_exact_small_integers(M, K, N, layout):
    vals, meta, b, ref = _operands(M, K, N, M + K + N, exact=True)
    got = _gpu(vals, meta, b, K, layout)
    np.testing.assert_array_equal(got, obf.from_f64(ref))


@pytest.mark.parametrize("layout", [elas.ELAS_B_NK, elas.ELAS_B_KN])
@pytest.mark.parametrize("M,K,N", SHAPES[3:])
def test_gaussian(M, K, N, layout):
    vals, meta, b, ref = _operands(M, K, N, 7 * M + K, exact=False)
    got = obf.to_f64(_gpu(vals, meta, b, K, layout))
    assert rel_fro(got, ref) < 5e-3
    # elementwise: fp32 accumulation of K products errs by at most
    # K 2^-24 sum|a||b| (standard summation bound), then one bf16 rounding
    # adds at most 2^-8 of the accumulator's magnitude
    dense, _ = osp.decompress(obf.to_f64(vals), meta, K)
    e = K * 2.0 ** -24 * (np.abs(dense) @ np.abs(obf.to_f64(b)))
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * (np.abs(ref) + e) + e + 2.0 ** -133)


def test_zero_rows_is_noop():
    K, N = 64, 16
    c = elas.elas_spmm_24(torch.zeros((0, 32), dtype=torch.bfloat16, device="cuda:0"),
                          torch.zeros((0, 8), dtype=torch.uint8, device="cuda:0"), K,
                          torch.zeros((N, K), dtype=torch.bfloat16, device="cuda:0"), elas.ELAS_B_NK)
    torch.cuda.synchronize()
    assert c.shape == (0, N)


def _random_shapes(n, seed):
    g = np.random.default_rng(seed)
    return [(int(g.integers(1, 1200)), 8 * int(g.integers(1, 400)), 8 * int(g.integers(1, 80))) for _ in range(n)]


@pytest.mark.parametrize("layout", [elas.ELAS_B_NK, elas.ELAS_B_KN])
@pytest.mark.parametrize("M,K,N", _random_shapes(10, 2026))
def test_random_shapes_exact(M, K, N, layout):
    """Seeded random M (any), K and N (multiples of 8): bit-exact on small integers."""
    vals, meta, b, ref = _operands(M, K, N, M + 3 * K + N, exact=True)
    got = _gpu(vals, meta, b, K, layout)
    np.testing.assert_array_equal(got, obf.from_f64(ref))


@pytest.mark.parametrize("M,K,N", [(24832, 2736, 512), (49408, 5464, 256)])
def test_exact_persistent_256_tiles(M, K, N):
    """M large enough for at least 192 tiles of 256 x 256, so the product runs
    the persistent 256 x 256 smfmac configuration on the row-layout 2:4
    operand (smaller problems take 128 x 128 tiles): bit-exact on small
    integers in both layouts of B."""
    vals, meta, b, ref = _operands(M, K, N, M + K + N, exact=True)
    want = obf.from_f64(ref)
    for layout in (elas.ELAS_B_NK, elas.ELAS_B_KN):
        got = _gpu(vals, meta, b, K, layout)
        np.testing.assert_array_equal(got, want, err_msg=f"layout {layout}")
