"""Seeded sweep of forward + backward over random shapes against the oracle:
token counts from 1 to a few thousand (ragged against every tile size),
d, d_ff and r random multiples of 8 (d_ff often not a multiple of 64, so the
compressed rows are padded), in every activation mode, plus the fused forward
on its supported shapes.  Same gates as the other parity tests."""
import numpy as np
import pytest

import paper_2605_03667_amd as elas
from oracle import ffn as offn
from synthetic import ffn_inputs
from tests.test_gpu_ffn import compare, run_gpu

pytestmark = pytest.mark.gpu


def _shapes(n, seed):
    g = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        T = int(g.choice([1, 2, 31, 33, 255, 257, 511, 777, 1025, 2049, 3001]))
        d = 8 * int(g.integers(1, 65))        # 8 .. 512
        F = 8 * int(g.integers(1, 161))       # 8 .. 1280
        r = 8 * int(g.integers(1, 41))        # 8 .. 320
        out.append((T, d, F, r))
    return out


@pytest.mark.parametrize("mode", ["sparse", "dense", "ste"])
@pytest.mark.parametrize("T,d,F,r", _shapes(24, 2026))
def test_random_shapes(T, d, F, r, mode):
    bits = ffn_inputs(T, d, F, r, seed_base=T + d + F + r)
    f, b = offn.run(bits, sparse=(mode != "dense"), ste=(mode == "ste"))
    compare(run_gpu(bits, mode=mode), f, b, bits, mode=mode)


def _fused_shapes(n, seed):
    g = np.random.default_rng(seed)
    return [(int(g.choice([1, 40, 97, 1000, 2500])), 64 * int(g.integers(1, 17)), 8 * int(g.integers(1, 161)),
             int(g.choice([128, 256]))) for _ in range(n)]


@pytest.mark.parametrize("T,d,F,r", _fused_shapes(6, 7))
def test_random_shapes_fused(T, d, F, r):
    bits = ffn_inputs(T, d, F, r, seed_base=T + d + F + r + 1)
    f, b = offn.run(bits)
    compare(run_gpu(bits, fwd_flags=elas.ELAS_FWD_FUSED), f, b, bits)
