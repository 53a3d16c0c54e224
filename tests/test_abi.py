"""The C-ABI library on the host: it loads, exports every function that
include/elas.h declares, reports sizes, and rejects every invalid argument
with the documented status code before launching anything (so these calls
never touch a GPU)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2605_03667_amd as elas

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "elas.h")

pytestmark = pytest.mark.skipif(not os.path.exists(elas.LIB_PATH), reason="libelas.so not built")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(elas_[a-z0-9_]+)\s*\(", text)))


def _defines():
    out = {}
    for m in re.finditer(r"#define\s+(ELAS_[A-Z0-9_]+)\s+([0-9]+)u?", open(HEADER).read()):
        out[m.group(1)] = int(m.group(2))
    return out


def test_exports_every_declared_symbol():
    names = _declared()
    assert len(names) == 16, names
    lib = ctypes.CDLL(elas.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) <= set(elas._SIGNATURES)


def test_binding_constants_match_header():
    d = _defines()
    assert d["ELAS_SPARSIFY_RELU2"] == elas.ELAS_SPARSIFY_RELU2
    assert d["ELAS_SPARSIFY_RAW"] == elas.ELAS_SPARSIFY_RAW
    assert d["ELAS_B_KN"] == elas.ELAS_B_KN and d["ELAS_B_NK"] == elas.ELAS_B_NK
    assert d["ELAS_MODE_SPARSE24"] == elas.ELAS_MODE_SPARSE24 and d["ELAS_MODE_DENSE"] == elas.ELAS_MODE_DENSE
    assert d["ELAS_BWD_STE"] == elas.ELAS_BWD_STE
    assert d["ELAS_FACTORS_AB"] == elas.ELAS_FACTORS_AB
    for k, v in elas._STATUS.items():
        assert d[v] == k


def test_pitches_and_workspace_sizes():
    assert elas.elas_vals_ld(5464) == 2752 and elas.elas_meta_ld(5464) == 688
    assert elas.elas_vals_ld(64) == 32 and elas.elas_meta_ld(64) == 8
    assert elas.elas_vals_ld(8) == 32 and elas.elas_meta_ld(0) == 0
    lib = elas.lib()
    assert lib.elas_status_string(2) == b"ELAS_ERR_SHAPE"
    w = elas.elas_lowrank_ffn_fwd_workspace_bytes(65536, 2048, 5464, 512)
    assert w >= 2 * (512 * 2048 * 2 + 5504 * 512 * 2)
    wb = elas.elas_lowrank_ffn_bwd_workspace_bytes(65536, 2048, 5464, 512)
    assert wb >= 65536 * (512 * 2 * 2 + 2752 * 2)
    wd = elas.elas_lowrank_ffn_bwd_workspace_bytes(65536, 2048, 5464, 512, elas.ELAS_MODE_DENSE)
    ws = elas.elas_lowrank_ffn_bwd_workspace_bytes(65536, 2048, 5464, 512, elas.ELAS_BWD_STE)
    assert wd >= 65536 * (512 * 2 * 2 + 5464 * 2) and ws >= wd + 65536 * 5464 * 2
    assert elas.elas_spmm_24_workspace_bytes(10, 64, 32, elas.ELAS_B_NK) == 0
    assert elas.elas_spmm_24_workspace_bytes(10, 64, 32, elas.ELAS_B_KN) >= 64 * 32 * 2


FAKE = ctypes.c_void_p(0x10000)        # aligned, never dereferenced: every call below fails validation
MIS = ctypes.c_void_p(0x10008)


def _err(rc):
    return rc, elas.lib().elas_last_error().decode()


def test_sparsify_validation():
    L = elas.lib()
    assert _err(L.elas_sparsify_24(None, 4, 8, 0, FAKE, FAKE, None))[0] == 1
    assert _err(L.elas_sparsify_24(FAKE, 4, 12, 0, FAKE, FAKE, None))[0] == 2
    assert _err(L.elas_sparsify_24(FAKE, -1, 8, 0, FAKE, FAKE, None))[0] == 2
    assert _err(L.elas_sparsify_24(FAKE, 4, 0, 0, FAKE, FAKE, None))[0] == 2
    assert _err(L.elas_sparsify_24(MIS, 4, 8, 0, FAKE, FAKE, None))[0] == 3
    rc, msg = _err(L.elas_sparsify_24(FAKE, 4, 8, 6, FAKE, FAKE, None))
    assert rc == 5 and "flags" in msg


def test_spmm_validation():
    L = elas.lib()
    assert L.elas_spmm_24(FAKE, FAKE, 4, 64, FAKE, 32, 2, FAKE, None, 0, None) == 5
    assert L.elas_spmm_24(FAKE, FAKE, 4, 60, FAKE, 32, 1, FAKE, None, 0, None) == 2
    assert L.elas_spmm_24(FAKE, FAKE, 4, 64, FAKE, 30, 1, FAKE, None, 0, None) == 2
    assert L.elas_spmm_24(FAKE, None, 4, 64, FAKE, 32, 1, FAKE, None, 0, None) == 1
    assert L.elas_spmm_24(FAKE, FAKE, 4, 64, FAKE, 32, 1, MIS, None, 0, None) == 3
    # B given as [K x N] needs a workspace for its transpose
    assert L.elas_spmm_24(FAKE, FAKE, 4, 64, FAKE, 32, 0, FAKE, None, 0, None) == 4


def _fwd(L, T=16, d=32, F=64, r=16, flags=0, ws=None, wsb=None, x=FAKE, y=FAKE):
    if wsb is None:
        wsb = L.elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r, flags)
    return L.elas_lowrank_ffn_fwd(x, FAKE, FAKE, FAKE, FAKE, T, d, F, r, flags, y, FAKE, FAKE, FAKE, FAKE,
                                  ws, wsb, None)


def test_fwd_validation():
    L = elas.lib()
    assert _fwd(L, flags=1) == 5
    assert _fwd(L, flags=4) == 5                # STE is a backward-only flag
    assert _fwd(L, flags=64) == 5
    assert _fwd(L, flags=16 | 32) == 5         # fused and unfused at once
    assert _fwd(L, flags=16 | 2) == 5          # the fused forward is sparse-mode only
    assert _fwd(L, flags=16) == 2              # d = 32, r = 16: no fused kernel for that shape
    assert _fwd(L, d=64, r=128, flags=16) == 1  # supported shape: on to the pointer checks (x is fake, y fine)
    # pre-arranged factors need no factor copies in the workspace
    assert (L.elas_lowrank_ffn_fwd_workspace_bytes(65536, 2048, 5464, 512, 8)
            < L.elas_lowrank_ffn_fwd_workspace_bytes(65536, 2048, 5464, 512, 0))
    assert _fwd(L, d=12) == 2
    assert _fwd(L, F=60) == 2
    assert _fwd(L, r=0) == 2
    assert _fwd(L, T=-3) == 2
    assert _fwd(L, x=None) == 1
    assert _fwd(L, y=MIS) == 3
    assert _fwd(L, ws=FAKE, wsb=1) == 4          # too small
    assert _fwd(L, ws=None) == 1                 # enough bytes claimed but NULL


def test_bwd_validation():
    L = elas.lib()
    T, d, F, r = 16, 32, 64, 16
    need = L.elas_lowrank_ffn_bwd_workspace_bytes(T, d, F, r, 0)

    def call(**kw):
        a = dict(dy=FAKE, flags=0, d=d, ws=FAKE, wsb=need, dV_down=FAKE)
        a.update(kw)
        return L.elas_lowrank_ffn_bwd(a["dy"], FAKE, FAKE, FAKE, FAKE, FAKE, T, a["d"], F, r, a["flags"],
                                      FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, a["dV_down"],
                                      a["ws"], a["wsb"], None)
    assert call(flags=8) == 5                   # unknown bit
    assert call(flags=6) == 5                   # STE needs the sparse forward
    assert call(d=20) == 2
    assert call(dy=None) == 1
    assert call(dV_down=MIS) == 3
    assert call(wsb=need - 1) == 4


def test_fullrank_validation():
    L = elas.lib()

    def call(**kw):
        a = dict(x=FAKE, T=16, d=32, F=64, y=FAKE)
        a.update(kw)
        return L.elas_fullrank_ffn_fwd(a["x"], FAKE, FAKE, a["T"], a["d"], a["F"], a["y"], FAKE, None)
    assert call(d=12) == 2
    assert call(F=60) == 2
    assert call(T=-1) == 2
    assert call(x=None) == 1
    assert call(y=MIS) == 3
    assert call(T=0, x=None, y=None) == 0     # no tokens: nothing inspected


def test_tiled_layout_helpers():
    """The test-side conversion between row-major and the tiled layout of the
    saved S matches the index formula the header states: entry j of row t at
    (t // 256) * 256 * ld + (j // bw) * R * bw + (t % 256) * bw + j % bw, with
    R the rows of t's block of 256 (ragged last block included)."""
    from tests.helpers import tile, untile

    def index(t, j, T, ld, bw):
        tb = t // 256
        R = min(256, T - 256 * tb)
        return 256 * tb * ld + (j // bw) * R * bw + (t % 256) * bw + j % bw

    for T in (1, 7, 256, 300, 513):
        for ld, bw in ((64, 32), (96, 32), (16, 8), (24, 8)):
            a = np.arange(T * ld).reshape(T, ld)
            flat = np.empty(T * ld, dtype=a.dtype)
            for t in range(T):
                for j in range(ld):
                    flat[index(t, j, T, ld, bw)] = a[t, j]
            assert np.array_equal(tile(a, bw), flat)
            assert np.array_equal(untile(flat.reshape(T, ld), T, ld, bw), a)


def test_timing_filter_is_host_only():
    """elas_timing_only touches no device: it can be set and cleared on CPU."""
    L = elas.lib()
    assert L.elas_timing_only(b"b3_dH_masked") == 0
    assert L.elas_timing_only(None) == 0
    assert L.elas_timing_only(b"") == 0

