"""The debug mode (ELAS_DEBUG_SYNC: synchronise after every kernel and report
failures by kernel) leaves every result unchanged, and the saved compressed S
reads back in canonical form through the library's converters exactly as the
test formula untiles it."""
import numpy as np
import pytest
import torch

import paper_2605_03667_amd as elas
from synthetic import ffn_inputs
from tests.helpers import dev_bf16, host_bits, untile

pytestmark = pytest.mark.gpu


def _run(bits):
    t = {k: dev_bf16(v) for k, v in bits.items()}
    fwd = elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"])
    bwd = elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], fwd)
    sp = elas.elas_sparsify_24(t["x"])
    torch.cuda.synchronize()
    out = {k: v.view(torch.int16).cpu().numpy() if v.dtype == torch.bfloat16 else v.cpu().numpy()
           for k, v in list(fwd.items()) + list(bwd.items()) if v is not None}
    out["sp_vals"], out["sp_meta"] = host_bits(sp[0]), sp[1].cpu().numpy()
    return out


def test_debug_sync_same_results():
    bits = ffn_inputs(700, 136, 1000, 72, seed_base=17)
    ref = _run(bits)
    prev = elas.elas_debug_sync(True)
    try:
        got = _run(bits)
    finally:
        elas.elas_debug_sync(prev)
    for k in ref:
        np.testing.assert_array_equal(got[k], ref[k], err_msg=k)


def test_canonical_readback_of_saved_s():
    T, d, F, r = 600, 64, 200, 32
    bits = ffn_inputs(T, d, F, r, seed_base=23)
    t = {k: dev_bf16(v) for k, v in bits.items()}
    fwd = elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"])
    torch.cuda.synchronize()
    vals = elas.elas_vals_to_canonical(fwd["s_vals"].view(torch.int16), T, F)
    meta = elas.elas_meta_to_canonical(fwd["s_meta"], T, F)
    want_v = host_bits(untile(fwd["s_vals"], T, fwd["s_vals"].shape[1], 32))[:, : F // 2]
    want_m = untile(fwd["s_meta"], T, fwd["s_meta"].shape[1], 8).cpu().numpy()[:, : F // 8]
    np.testing.assert_array_equal(vals, want_v)
    np.testing.assert_array_equal(meta, want_m)
