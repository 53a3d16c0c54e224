"""bench.py's accounting (CPU): algorithmic FLOP and bytes per launch at the
1B shape, the bound each kernel falls under, and the one-GPU contract."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

T, d, F, r = 65536, 2048, 5464, 512


def test_flops_of_the_products():
    # dense products 2 FLOP per multiply-add; a 2:4 side counts its kept half
    assert bench.algorithmic_flops("k1_up_gemm", T, d, F, r) == 2 * T * d * r
    assert bench.algorithmic_flops("k3_spmm_down", T, d, F, r) == T * r * F
    assert bench.algorithmic_flops("k2_up_relu2_sparsify", T, d, F, r) == 2 * T * r * F
    # the twelve products of the masked step: six dense d x r products, k2 over the whole of d_ff,
    # and k3, b3, b4, b5, b6 on the kept half
    tags = ["k1_up_gemm", "k2_up_relu2_sparsify", "k3_spmm_down", "k4_down_gemm", "b1_dZ", "b2_dV_down",
            "b3_dH_masked", "b4_dU_down", "b5_spmm_dP", "b6_dV_up", "b7_dU_up", "b8_dx"]
    total = sum(bench.algorithmic_flops(t, T, d, F, r) for t in tags)
    assert total == 6 * 2 * T * d * r + 2 * T * r * F + 5 * T * r * F
    # the executed count of the smfmac and expanded 2:4 products is the dense one over padded d_ff
    assert bench.executed_flops("b4_dU_down", T, d, F, r) == 2 * T * r * 5504
    assert bench.executed_flops("b3_dH_ste", T, d, F, r) == 4 * T * r * 5504
    assert bench.algorithmic_flops("splitk_reduce", T, d, F, r) is None


def test_bytes_and_bound():
    # compressed S: d_ff/2 bf16 values and d_ff/8 code bytes per token (1.125 B per feature)
    S = T * F * 1.125
    assert bench.algorithmic_bytes("k3_spmm_down", T, d, F, r) == S + 2 * (F * r + T * r)
    b3 = bench.roofline_of("b3_dH_masked", T, d, F, r, 500e-6)
    ridge = bench.PEAK_BF16_TFLOPS * 1e12 / (bench.PEAK_HBM_GBS * 1e9)
    assert b3["intensity_flop_per_byte"] < ridge and b3["bound"] == "hbm" and b3["unit"] == "GB/s"
    assert b3["achieved"] == pytest.approx(b3["alg_bytes_per_launch"] / 500e-6 / 1e9, rel=1e-3)
    assert b3["frac"] == pytest.approx(b3["achieved"] / bench.PEAK_HBM_GBS, rel=1e-3)
    k1 = bench.roofline_of("k1_up_gemm", T, d, F, r, 130e-6)
    assert k1["intensity_flop_per_byte"] > ridge and k1["bound"] == "mfma" and k1["unit"] == "TFLOP/s"
    assert k1["achieved"] == pytest.approx(2 * T * d * r / 130e-6 / 1e12, rel=1e-3)
    assert bench.roofline_of("splitk_reduce", T, d, F, r, 1e-5) is None


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert p.returncode == 2 and "one GPU" in p.stderr and p.stdout == ""
