"""elas_lowrank_ffn_fwd_noalloc (the forward whose workspace is the library's
static device scratch) against elas_lowrank_ffn_fwd (caller's workspace):
every output bit-identical, on two calls in a row, the second with a smaller
input, in the 2:4 and dense modes and with the fused launch; and shapes whose
workspace exceeds the scratch are refused before anything is launched."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2605_03667_amd as elas
from synthetic import config_inputs, ffn_inputs
from tests.helpers import dev_bf16

pytestmark = pytest.mark.gpu


def _both(bits, flags):
    t = {k: dev_bf16(v) for k, v in bits.items()}
    ref = elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], flags=flags)
    # fill the outputs with garbage first, so that nothing passes by leftover contents
    got = {k: (torch.full_like(v, -7) if v is not None else None) for k, v in ref.items()}
    elas.elas_lowrank_ffn_fwd_noalloc(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], flags=flags, out=got)
    torch.cuda.synchronize()
    for k in ref:
        if ref[k] is None:
            continue
        a = ref[k].view(torch.int16) if ref[k].dtype == torch.bfloat16 else ref[k]
        b = got[k].view(torch.int16) if got[k].dtype == torch.bfloat16 else got[k]
        assert torch.equal(a, b), k


@pytest.mark.parametrize("flags", [0, 2, 16])
def test_noalloc_matches_workspace_forward_twice(flags):
    # first call: the 1B shape at 4096 tokens (about 15 MB of transposed factors in the scratch);
    # second call, smaller: 512 tokens of the 60M shape (small-T split-K partials in the scratch)
    if flags == 16:   # the fused forward needs d <= 1024
        first, second = config_inputs("llama350m", T=4096), config_inputs("llama60m", T=512)
    else:
        first, second = config_inputs("llama1b", T=4096), config_inputs("llama60m", T=512)
    _both(first, flags)
    _both(second, flags)


def test_noalloc_small_token_counts_1b():
    """At 256 tokens the 1B forward splits K over the CUs: its fp32 partials
    live in the scratch too (the largest forward workspace, about 31 MB)."""
    need = elas.elas_lowrank_ffn_fwd_workspace_bytes(256, 2048, 5464, 512, 0)
    assert need <= elas.elas_noalloc_scratch_bytes()
    _both(config_inputs("llama1b", T=256), 0)
    _both(ffn_inputs(77, 64, 136, 24, seed_base=3), 0)


def test_noalloc_refuses_oversized_shapes():
    L = elas.lib()
    fake = ctypes.c_void_p(0x10000)
    T, d, F, r = 1024, 65536, 65536, 512
    assert elas.elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r, 0) > elas.elas_noalloc_scratch_bytes()
    rc = L.elas_lowrank_ffn_fwd_noalloc(*([fake] * 5), T, d, F, r, 0, *([fake] * 5), None)
    assert rc == 4 and b"static scratch" in L.elas_last_error()
