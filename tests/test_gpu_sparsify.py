"""elas_sparsify_24 on the GPU against the oracle: bit-exact kept values and
metadata on the same bf16 input (Algorithm 1 with Eq. 2 in front), for both
selection modes, several value distributions, ragged shapes and the full
350M-shape workload (sampled rows), plus the padding content."""
import numpy as np
import pytest
import torch

import paper_2605_03667_amd as elas
from oracle import sparsify as osp
from synthetic import SPARSIFY_SHAPE, h_input
from tests.helpers import check_padding, dev_bf16, host_bits, meta_ld, vals_ld

pytestmark = pytest.mark.gpu


def _run(h_bits, mode):
    h = dev_bf16(h_bits)
    vals, meta = elas.elas_sparsify_24(h, mode)
    torch.cuda.synchronize()
    return host_bits(vals), meta.cpu().numpy()


def _compare(h_bits, mode, rows=None):
    M, N = h_bits.shape
    vals, meta = _run(h_bits, mode)
    assert vals.shape == (M, vals_ld(N)) and meta.shape == (M, meta_ld(N))
    check_padding(vals, meta, N)
    sel = slice(None) if rows is None else rows
    rv, rm = osp.sparsify24_bf16(h_bits[sel], mode)
    np.testing.assert_array_equal(meta[sel][:, : N // 8], rm)
    np.testing.assert_array_equal(vals[sel][:, : N // 2], rv)


@pytest.mark.parametrize("mode", [osp.RELU2, osp.RAW])
@pytest.mark.parametrize("shape", [(1, 8), (3, 16), (5, 24), (7, 72), (64, 1376), (33, 5464), (129, 2736),
                                   (2, 4104)])
def test_shapes(shape, mode):
    _compare(h_input(*shape, seed=shape[0] * 7 + shape[1]), mode)


@pytest.mark.parametrize("mode", [osp.RELU2, osp.RAW])
@pytest.mark.parametrize("mu,levels", [(0.0, None), (-0.994, None), (-2.054, None), (0.0, 8), (0.5, 3)])
def test_distributions(mu, levels, mode):
    """N(0,1), the 84 % and 98 % post-ReLU^2 sparsity the paper reports after
    warm-up, and quantised inputs that force ties."""
    _compare(h_input(257, 1376, seed=11, mu=mu, levels=levels), mode)


def test_special_values():
    """Zeros of both signs, infinities, NaNs, the largest finite bf16, the
    smallest subnormal and powers of two at both ends of the fp32 range.  All
    of them square exactly or saturate the same way on both sides, so the
    ReLU^2 output is bit-exact; NaN ranks as 0 (relu(NaN) = 0)."""
    specials = np.array([0x0000, 0x8000, 0x7F80, 0xFF80, 0x7FC0, 0xFFC0, 0x7F7F, 0xFF7F,
                         0x0001, 0x8001, 0x0080, 0x3F80, 0xBF80, 0x2000, 0x5F80, 0x1F80], dtype=np.uint16)
    g = np.random.default_rng(3)
    h = g.choice(specials, size=(64, 256)).astype(np.uint16)
    _compare(h, osp.RELU2)
    # the raw mode ranks |h|; NaN is outside its domain and is replaced by 1.0
    hr = np.where((h & 0x7FFF) > 0x7F80, np.uint16(0x3F80), h).astype(np.uint16)
    _compare(hr, osp.RAW)


def test_full_350m_shape_sampled_rows():
    M, N = SPARSIFY_SHAPE
    h = h_input(M, N, seed=2)
    rows = np.unique(np.concatenate([[0, 1, M - 1], np.random.default_rng(0).integers(0, M, 509)]))
    _compare(h, osp.RELU2, rows=rows)


def test_empty_rows_is_noop():
    h = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda:0")
    vals, meta = elas.elas_sparsify_24(h)
    torch.cuda.synchronize()
    assert vals.shape == (0, 32) and meta.shape == (0, 8)


def test_bad_shape_raises():
    h = torch.zeros((4, 12), dtype=torch.bfloat16, device="cuda:0")
    with pytest.raises(elas.ElasError) as e:
        elas.elas_sparsify_24(h, vals=torch.empty((4, 32), dtype=torch.bfloat16, device="cuda:0"),
                              meta=torch.empty((4, 8), dtype=torch.uint8, device="cuda:0"))
    assert e.value.code == 2
