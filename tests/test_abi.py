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
    assert len(names) == 21, names
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
    assert wd >= 65536 * (512 * 2 * 2 + 5464 * 2)
    # straight-through: dZ, dense dH, dP and V_up^T; relu(h) stays in the dH kernel's registers
    assert ws >= 65536 * (512 * 2 * 2 + 5464 * 2) + 5504 * 512 * 2 and ws < wd + 65536 * 5464 * 2
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



def _cpu(shape, dtype=None):
    import torch
    return torch.zeros(shape, dtype=dtype or torch.bfloat16)


def test_binding_rejects_mismatched_shapes():
    """The binding checks every tensor's shape against the sizes it passes to
    the C ABI (which cannot check buffer sizes) before taking any pointer,
    so a wrong size raises instead of reading or writing out of bounds.
    Nothing is launched: the tensors are on the CPU."""
    import torch
    T, d, F, r = 8, 16, 24, 8
    ldv, ldm = elas.elas_vals_ld(F), elas.elas_meta_ld(F)
    x, dy = _cpu((T, d)), _cpu((T, d))
    fac = {"U_up": _cpu((d, r)), "V_up": _cpu((r, F)), "U_down": _cpu((F, r)), "V_down": _cpu((r, d))}
    sparse_saved = {"y": _cpu((T, d)), "P": _cpu((T, r)), "s_vals": _cpu((T, ldv)),
                    "s_meta": _cpu((T, ldm), torch.uint8), "Z": _cpu((T, r))}
    dense_saved = dict(sparse_saved, s_vals=_cpu((T, F)), s_meta=None)
    f32 = torch.float32
    grads = {"dx": _cpu((T, d)), "dU_up": _cpu((d, r), f32), "dV_up": _cpu((r, F), f32),
             "dU_down": _cpu((F, r), f32), "dV_down": _cpu((r, d), f32)}

    def raises(match, fn, *a, **k):
        with pytest.raises(ValueError, match=match):
            fn(*a, **k)

    bwd = elas.elas_lowrank_ffn_bwd
    # a sparse forward's saved tensors with the dense flag (s_vals half as wide), and vice versa
    raises("s_vals \\(dense mode\\)", bwd, dy, x, *fac.values(), sparse_saved, flags=elas.ELAS_MODE_DENSE, grads=grads)
    raises("s_vals \\(2:4 mode\\)", bwd, dy, x, *fac.values(), dense_saved, flags=0, grads=grads)
    raises("s_meta", bwd, dy, x, *fac.values(), dict(sparse_saved, s_meta=_cpu((T, ldm - 8), torch.uint8)), grads=grads)
    for k in grads:
        bad = dict(grads, **{k: _cpu((grads[k].shape[0] + 1, grads[k].shape[1]), grads[k].dtype)})
        raises(k, bwd, dy, x, *fac.values(), sparse_saved, grads=bad)
    raises("dy", bwd, _cpu((T + 1, d)), x, *fac.values(), sparse_saved, grads=grads)
    raises("U_down", bwd, dy, x, fac["U_up"], fac["V_up"], _cpu((F + 8, r)), fac["V_down"], sparse_saved, grads=grads)
    fwd = elas.elas_lowrank_ffn_fwd
    raises("V_down", fwd, x, fac["U_up"], fac["V_up"], fac["U_down"], _cpu((r, d + 8)), out=sparse_saved)
    raises("Z", fwd, x, *fac.values(), out=dict(sparse_saved, Z=_cpu((T, r + 8))))
    raises("s_vals \\(dense mode\\)", fwd, x, *fac.values(), flags=elas.ELAS_MODE_DENSE, out=sparse_saved)
    # factors given as A, B (transposed) without the flag
    raises("U_up", fwd, x, *(t.t().contiguous() for t in fac.values()), out=sparse_saved)
    # standalone calls
    raises("vals", elas.elas_sparsify_24, _cpu((T, F)), vals=_cpu((T, ldv - 8)), meta=_cpu((T, ldm), torch.uint8))
    raises("a_vals", elas.elas_spmm_24, _cpu((T, F // 2)), _cpu((T, ldm), torch.uint8), F, _cpu((r, F)), elas.ELAS_B_NK)
    raises("b", elas.elas_spmm_24, _cpu((T, ldv)), _cpu((T, ldm), torch.uint8), F, _cpu((r, F)), elas.ELAS_B_KN)
    raises("c", elas.elas_spmm_24, _cpu((T, ldv)), _cpu((T, ldm), torch.uint8), F, _cpu((r, F)), elas.ELAS_B_NK,
           c=_cpu((T, r + 8)))
    raises("W_down", elas.elas_fullrank_ffn_fwd, x, _cpu((F, d)), _cpu((F, d)))


def test_canonical_converters_match_the_tiled_formula():
    """elas_meta_to_canonical / elas_vals_to_canonical undo the tiled layout
    of include/elas.h: checked against the independent test formula
    (tests/helpers.untile) on random contents, with a ragged last row block,
    and padding columns dropped."""
    from tests.helpers import tile
    g = np.random.default_rng(3)
    for M, N in [(1, 8), (255, 64), (600, 5464), (513, 200)]:
        ldv, ldm = elas.elas_vals_ld(N), elas.elas_meta_ld(N)
        rows_v = g.integers(0, 1 << 16, (M, ldv), dtype=np.uint16)
        rows_m = g.integers(0, 256, (M, ldm), dtype=np.uint8)
        tv, tm = tile(rows_v, 32).reshape(M, ldv), tile(rows_m, 8).reshape(M, ldm)
        np.testing.assert_array_equal(elas.elas_vals_to_canonical(tv, M, N), rows_v[:, : N // 2])
        np.testing.assert_array_equal(elas.elas_meta_to_canonical(tm, M, N), rows_m[:, : N // 8])
    L = elas.lib()
    assert L.elas_meta_to_canonical(None, 0, 64, None) == 0
    assert L.elas_meta_to_canonical(None, 4, 64, None) == elas._STATUS_CODE["ELAS_ERR_NULL"]
    assert L.elas_vals_to_canonical(FAKE, 4, 12, FAKE) == elas._STATUS_CODE["ELAS_ERR_SHAPE"]


def test_debug_sync_switch():
    prev = elas.elas_debug_sync(None)
    assert elas.elas_debug_sync(True) == prev
    assert elas.elas_debug_sync(None) is True
    assert elas.elas_debug_sync(False) is True
    assert elas.elas_debug_sync(prev) is False
