"""The entry points are capture-safe: a forward + backward captured in a HIP
graph (torch.cuda.CUDAGraph) and replayed several times, with eager work and
synchronisations between the replays, reproduces the eager results bit for
bit (the library allocates nothing and enqueues only kernels on the caller's
stream)."""
import numpy as np
import pytest
import torch

import paper_2605_03667_amd as elas
from synthetic import config_inputs, ffn_inputs
from tests.helpers import dev_bf16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,T", [(None, 300), ("llama1b", 512)])
@pytest.mark.parametrize("mode", ["sparse", "dense", "ste", "fused"])
def test_graph_replays_match_eager(name, T, mode):
    if mode == "fused":   # the fused forward's shapes: r = 128 (the 60M model instead of 1B)
        bits = config_inputs("llama60m", T=T) if name else ffn_inputs(T, 128, 264, 128, seed_base=9)
    else:
        bits = config_inputs(name, T=T) if name else ffn_inputs(T, 128, 264, 32, seed_base=9)
    t = {k: dev_bf16(v) for k, v in bits.items()}
    T, d = bits["x"].shape
    r, F = bits["V_up"].shape
    fflags = {"sparse": 0, "ste": 0, "dense": elas.ELAS_MODE_DENSE, "fused": elas.ELAS_FWD_FUSED}[mode]
    bflags = {"sparse": 0, "ste": elas.ELAS_BWD_STE, "dense": elas.ELAS_MODE_DENSE, "fused": 0}[mode]
    saved = elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], flags=fflags)
    grads = elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], saved,
                                      flags=bflags)
    wsf = torch.empty(max(1, elas.elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r, fflags)), dtype=torch.uint8,
                      device="cuda:0")
    wsb = torch.empty(max(1, elas.elas_lowrank_ffn_bwd_workspace_bytes(T, d, F, r, bflags)), dtype=torch.uint8,
                      device="cuda:0")

    def step():
        elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], flags=fflags, out=saved,
                                  workspace=wsf)
        elas.elas_lowrank_ffn_bwd(t["dY"], t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], saved,
                                  flags=bflags, grads=grads, workspace=wsb)

    step()
    torch.cuda.synchronize()
    outs = {k: v for k, v in list(saved.items()) + list(grads.items()) if v is not None}
    ref = {k: v.clone() for k, v in outs.items()}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for v in outs.values():
            v.zero_()                     # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in outs.items():
            assert torch.equal(v, ref[k]), (rep, k)


@pytest.mark.parametrize("name,T", [(None, 300), ("llama1b", 512), ("llama1b", 4096)])
def test_graph_replays_noalloc_forward(name, T):
    """The no-allocation forward (its workspace the library's static scratch)
    captured in a graph with nothing but the caller's inputs and outputs:
    every replay, with eager work between them, equals the eager result and
    the workspace forward's, bit for bit."""
    bits = config_inputs(name, T=T) if name else ffn_inputs(T, 128, 264, 32, seed_base=19)
    t = {k: dev_bf16(v) for k, v in bits.items()}
    ref = elas.elas_lowrank_ffn_fwd(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"])
    out = {k: torch.empty_like(v) for k, v in ref.items()}

    def fwd():
        elas.elas_lowrank_ffn_fwd_noalloc(t["x"], t["U_up"], t["V_up"], t["U_down"], t["V_down"], out=out)

    fwd()                                   # first call on the device: looks the scratch up, outside the capture
    torch.cuda.synchronize()
    for k in ref:
        assert torch.equal(out[k], ref[k]), k
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fwd()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fwd()
    for rep in range(3):
        for v in out.values():
            v.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(out[k], ref[k]), (rep, k)
