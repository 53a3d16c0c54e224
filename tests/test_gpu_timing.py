"""The diagnostics timing API that bench.py relies on: with every launch
recorded, one forward + backward reports each kernel tag of the launch
sequence; with elas_timing_only(tag), only that tag's launches are recorded;
the outputs are the same with or without recording."""
import pytest
import torch

import paper_2605_03667_amd as elas
from synthetic import ffn_inputs
from tests.helpers import dev_bf16

pytestmark = pytest.mark.gpu


def _step(t, out=None):
    fwd = elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], out=out)
    bwd = elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], fwd)
    return fwd, bwd


def test_timing_all_and_filtered():
    t = {k: dev_bf16(v) for k, v in ffn_inputs(4096, 512, 1376, 128, seed_base=9).items()}
    ref_f, ref_b = _step(t)
    torch.cuda.synchronize()
    try:
        elas.elas_timing_only(None)
        elas.elas_timing_enable(True)
        f1, b1 = _step(t)
        torch.cuda.synchronize()
        elas.elas_timing_enable(False)
        every = elas.elas_timing_collect()
        for tag in ("k1_up_gemm", "k2_up_relu2_sparsify", "k3_spmm_down", "k4_down_gemm", "b3_dH_masked",
                    "b5_spmm_dP", "b8_dx"):
            assert every.get(tag, (0, 0.0))[0] == 1, (tag, every)
        assert all(ms > 0 for _, ms in every.values()), every

        elas.elas_timing_only("b3_dH_masked")
        elas.elas_timing_enable(True)
        f2, b2 = _step(t)
        torch.cuda.synchronize()
        elas.elas_timing_enable(False)
        only = elas.elas_timing_collect()
        assert list(only) == ["b3_dH_masked"] and only["b3_dH_masked"][0] == 1, only
    finally:
        elas.elas_timing_enable(False)
        elas.elas_timing_only(None)
    for f, b in ((f1, b1), (f2, b2)):
        assert torch.equal(f["y"].view(torch.int16), ref_f["y"].view(torch.int16))
        assert torch.equal(b["dx"].view(torch.int16), ref_b["dx"].view(torch.int16))
        assert torch.equal(b["dU_down"], ref_b["dU_down"])
