"""Python binding of libelas, the MI355X (gfx950) ELAS low-rank 2:4 FFN.

Thin ctypes wrapper over the C ABI declared in ``include/elas.h``: the
functions here carry the same names as the C entry points and only marshal
arguments (torch tensors -> device pointers and sizes, the current HIP stream,
output and workspace tensors).  Every step of the computation runs in the HIP
kernels of ``libelas.so``; there is no fallback: if the library is not built,
or a tensor is not on the GPU, the call raises.

bf16 tensors use ``torch.bfloat16``; the compressed 2:4 metadata uses
``torch.uint8``; weight gradients are ``torch.float32``.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "ElasError", "lib", "elas_vals_ld", "elas_meta_ld", "elas_sparsify_24", "elas_spmm_24",
    "elas_spmm_24_workspace_bytes", "elas_lowrank_ffn_fwd", "elas_lowrank_ffn_fwd_workspace_bytes",
    "elas_lowrank_ffn_bwd", "elas_lowrank_ffn_bwd_workspace_bytes", "elas_fullrank_ffn_fwd",
    "elas_timing_enable", "elas_timing_only", "elas_timing_collect", "elas_meta_to_canonical",
    "elas_vals_to_canonical", "elas_debug_sync", "elas_lowrank_ffn_fwd_noalloc", "elas_noalloc_scratch_bytes",
    "ELAS_SPARSIFY_RELU2", "ELAS_SPARSIFY_RAW", "ELAS_B_KN", "ELAS_B_NK", "ELAS_MODE_SPARSE24",
    "ELAS_MODE_DENSE", "ELAS_BWD_STE", "ELAS_FACTORS_AB", "ELAS_FWD_FUSED", "ELAS_FWD_UNFUSED",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libelas.so")

ELAS_SPARSIFY_RELU2 = 0
ELAS_SPARSIFY_RAW = 1
ELAS_B_KN = 0
ELAS_B_NK = 1
ELAS_MODE_SPARSE24 = 0
ELAS_MODE_DENSE = 2
ELAS_BWD_STE = 4
ELAS_FACTORS_AB = 8
ELAS_FWD_FUSED = 16
ELAS_FWD_UNFUSED = 32

_STATUS = {0: "ELAS_OK", 1: "ELAS_ERR_NULL", 2: "ELAS_ERR_SHAPE", 3: "ELAS_ERR_ALIGN",
           4: "ELAS_ERR_WORKSPACE", 5: "ELAS_ERR_FLAGS", 6: "ELAS_ERR_DEVICE"}


_STATUS_CODE = {v: k for k, v in _STATUS.items()}


class ElasError(RuntimeError):
    def __init__(self, code: int, detail: str):
        super().__init__(f"{_STATUS.get(code, code)}: {detail}")
        self.code = code
        self.detail = detail


_lib = None
_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_u32 = ctypes.c_uint32
_sz = ctypes.c_size_t

_SIGNATURES = {
    "elas_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "elas_last_error": ([], ctypes.c_char_p),
    "elas_vals_ld": ([_i64], _i64),
    "elas_meta_ld": ([_i64], _i64),
    "elas_sparsify_24": ([_p, _i64, _i64, _u32, _p, _p, _p], ctypes.c_int),
    "elas_spmm_24_workspace_bytes": ([_i64, _i64, _i64, ctypes.c_int], _sz),
    "elas_spmm_24": ([_p, _p, _i64, _i64, _p, _i64, ctypes.c_int, _p, _p, _sz, _p], ctypes.c_int),
    "elas_lowrank_ffn_fwd_workspace_bytes": ([_i64, _i64, _i64, _i64, _u32], _sz),
    "elas_lowrank_ffn_fwd": ([_p] * 5 + [_i64] * 4 + [_u32] + [_p] * 5 + [_p, _sz, _p], ctypes.c_int),
    "elas_noalloc_scratch_bytes": ([], _sz),
    "elas_lowrank_ffn_fwd_noalloc": ([_p] * 5 + [_i64] * 4 + [_u32] + [_p] * 5 + [_p], ctypes.c_int),
    "elas_lowrank_ffn_bwd_workspace_bytes": ([_i64, _i64, _i64, _i64, _u32], _sz),
    "elas_lowrank_ffn_bwd": ([_p] * 6 + [_i64] * 4 + [_u32] + [_p] * 4 + [_p] * 5 + [_p, _sz, _p],
                             ctypes.c_int),
    "elas_fullrank_ffn_fwd": ([_p] * 3 + [_i64] * 3 + [_p] * 3, ctypes.c_int),
    "elas_meta_to_canonical": ([_p, _i64, _i64, _p], ctypes.c_int),
    "elas_vals_to_canonical": ([_p, _i64, _i64, _p], ctypes.c_int),
    "elas_debug_sync": ([ctypes.c_int], ctypes.c_int),
    "elas_timing_enable": ([ctypes.c_int], ctypes.c_int),
    "elas_timing_only": ([ctypes.c_char_p], ctypes.c_int),
    "elas_timing_collect": ([], ctypes.c_int),
    "elas_timing_entry": ([ctypes.c_int, ctypes.c_char_p, ctypes.c_int, ctypes.POINTER(_i64),
                           ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
}


def lib() -> ctypes.CDLL:
    """The loaded libelas.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2605_03667_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGNATURES.items():
            f = getattr(handle, name)
            f.argtypes = args
            f.restype = res
        _lib = handle
    return _lib


def _check(rc: int) -> None:
    if rc != 0:
        raise ElasError(rc, lib().elas_last_error().decode())


def _shape(t: torch.Tensor | None, shape: tuple, name: str) -> None:
    """Raise unless tensor ``t`` has exactly ``shape``: the C ABI receives bare
    pointers and cannot check the size of a buffer, so a tensor of the wrong
    size would be read or written out of bounds.  Runs before any pointer is
    taken, so a wrong size is reported whatever the tensor's device."""
    if t is None:
        raise ValueError(f"{name} is required (shape {tuple(shape)})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _ptr(t: torch.Tensor | None, dtype: torch.dtype, name: str):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _workspace(nbytes: int, device: torch.device) -> torch.Tensor | None:
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def elas_vals_ld(N: int) -> int:
    return lib().elas_vals_ld(N)


def elas_meta_ld(N: int) -> int:
    return lib().elas_meta_ld(N)


def elas_sparsify_24(h: torch.Tensor, flags: int = ELAS_SPARSIFY_RELU2, vals: torch.Tensor | None = None,
                     meta: torch.Tensor | None = None):
    """2:4 sparsification of h [M, N] (bf16).  Returns (vals, meta)."""
    M, N = h.shape
    if vals is None:
        vals = torch.empty((M, elas_vals_ld(N)), dtype=torch.bfloat16, device=h.device)
    if meta is None:
        meta = torch.empty((M, elas_meta_ld(N)), dtype=torch.uint8, device=h.device)
    _shape(vals, (M, elas_vals_ld(N)), "vals")
    _shape(meta, (M, elas_meta_ld(N)), "meta")
    _check(lib().elas_sparsify_24(_ptr(h, torch.bfloat16, "h"), M, N, flags,
                                  _ptr(vals, torch.bfloat16, "vals"), _ptr(meta, torch.uint8, "meta"),
                                  _stream(h.device)))
    return vals, meta


def elas_spmm_24_workspace_bytes(M: int, K: int, N: int, b_layout: int) -> int:
    return lib().elas_spmm_24_workspace_bytes(M, K, N, b_layout)


def elas_spmm_24(a_vals: torch.Tensor, a_meta: torch.Tensor, K: int, b: torch.Tensor,
                 b_layout: int = ELAS_B_KN, c: torch.Tensor | None = None,
                 workspace: torch.Tensor | None = None) -> torch.Tensor:
    """C [M, N] = A B with A 2:4-compressed [M, K] (vals, meta) and B [K, N]
    (ELAS_B_KN) or [N, K] (ELAS_B_NK)."""
    M = a_vals.shape[0]
    if b.dim() != 2 or a_vals.dim() != 2:
        raise ValueError("a_vals and b must be 2-D")
    N = b.shape[1] if b_layout == ELAS_B_KN else b.shape[0]
    _shape(a_vals, (M, elas_vals_ld(K)), "a_vals")
    _shape(a_meta, (M, elas_meta_ld(K)), "a_meta")
    _shape(b, (K, N) if b_layout == ELAS_B_KN else (N, K), "b")
    if c is None:
        c = torch.empty((M, N), dtype=torch.bfloat16, device=a_vals.device)
    _shape(c, (M, N), "c")
    need = elas_spmm_24_workspace_bytes(M, K, N, b_layout)
    if workspace is None:
        workspace = _workspace(need, a_vals.device)
    _check(lib().elas_spmm_24(_ptr(a_vals, torch.bfloat16, "a_vals"), _ptr(a_meta, torch.uint8, "a_meta"), M, K,
                              _ptr(b, torch.bfloat16, "b"), N, b_layout, _ptr(c, torch.bfloat16, "c"),
                              _ptr(workspace, torch.uint8, "workspace"),
                              0 if workspace is None else workspace.numel(), _stream(a_vals.device)))
    return c


def _saved_shapes(saved: dict, T: int, d: int, F: int, r: int, dense: bool, with_y: bool) -> None:
    """Shapes of the forward's outputs (the backward's saved inputs) for the
    activation mode: dense s_vals [T, d_ff]; compressed s_vals
    [T, elas_vals_ld(d_ff)] and s_meta [T, elas_meta_ld(d_ff)]."""
    if with_y:
        _shape(saved.get("y"), (T, d), "y")
    _shape(saved.get("P"), (T, r), "P")
    _shape(saved.get("Z"), (T, r), "Z")
    if dense:
        _shape(saved.get("s_vals"), (T, F), "s_vals (dense mode)")
    else:
        _shape(saved.get("s_vals"), (T, elas_vals_ld(F)), "s_vals (2:4 mode)")
        _shape(saved.get("s_meta"), (T, elas_meta_ld(F)), "s_meta (2:4 mode)")


def elas_lowrank_ffn_fwd_workspace_bytes(T: int, d: int, d_ff: int, r: int, flags: int = 0) -> int:
    return lib().elas_lowrank_ffn_fwd_workspace_bytes(T, d, d_ff, r, flags)


def elas_lowrank_ffn_bwd_workspace_bytes(T: int, d: int, d_ff: int, r: int, flags: int = 0) -> int:
    return lib().elas_lowrank_ffn_bwd_workspace_bytes(T, d, d_ff, r, flags)


def elas_lowrank_ffn_fwd(x, U_up, V_up, U_down, V_down, flags: int = 0, out: dict | None = None,
                         workspace: torch.Tensor | None = None) -> dict:
    """Forward of the low-rank 2:4 FFN.  Returns dict(y, P, s_vals, s_meta, Z).

    s_vals [T, elas_vals_ld(d_ff)] and s_meta [T, elas_meta_ld(d_ff)] hold the
    compressed S in the tiled layout of include/elas.h (the tensors' shapes
    give the sizes, not row positions).  With ``flags=ELAS_MODE_DENSE`` s_vals
    is the dense row-major [T, d_ff] activation and s_meta is None.  With ``ELAS_FACTORS_AB`` the factors are passed transposed
    (U_up^T [r, d], V_up^T [d_ff, r], U_down^T [r, d_ff], V_down^T [d, r])."""
    T, d = x.shape
    ab = bool(flags & ELAS_FACTORS_AB)
    r = U_up.shape[0] if ab else U_up.shape[1]
    F = V_up.shape[0] if ab else V_up.shape[1]
    dev = x.device
    dense = bool(flags & ELAS_MODE_DENSE)
    for t, shp, name in ((U_up, (d, r), "U_up"), (V_up, (r, F), "V_up"), (U_down, (F, r), "U_down"),
                         (V_down, (r, d), "V_down")):
        _shape(t, shp[::-1] if ab else shp, name)
    if out is None:
        out = {
            "y": torch.empty((T, d), dtype=torch.bfloat16, device=dev),
            "P": torch.empty((T, r), dtype=torch.bfloat16, device=dev),
            "s_vals": torch.empty((T, F if dense else elas_vals_ld(F)), dtype=torch.bfloat16, device=dev),
            "s_meta": None if dense else torch.empty((T, elas_meta_ld(F)), dtype=torch.uint8, device=dev),
            "Z": torch.empty((T, r), dtype=torch.bfloat16, device=dev),
        }
    _saved_shapes(out, T, d, F, r, dense, with_y=True)
    need = elas_lowrank_ffn_fwd_workspace_bytes(T, d, F, r, flags)
    if workspace is None:
        workspace = _workspace(need, dev)
    bf = torch.bfloat16
    _check(lib().elas_lowrank_ffn_fwd(
        _ptr(x, bf, "x"), _ptr(U_up, bf, "U_up"), _ptr(V_up, bf, "V_up"), _ptr(U_down, bf, "U_down"),
        _ptr(V_down, bf, "V_down"), T, d, F, r, flags,
        _ptr(out["y"], bf, "y"), _ptr(out["P"], bf, "P"), _ptr(out["s_vals"], bf, "s_vals"),
        _ptr(out["s_meta"], torch.uint8, "s_meta"), _ptr(out["Z"], bf, "Z"),
        _ptr(workspace, torch.uint8, "workspace"), 0 if workspace is None else workspace.numel(),
        _stream(dev)))
    return out


def elas_noalloc_scratch_bytes() -> int:
    return lib().elas_noalloc_scratch_bytes()


def elas_lowrank_ffn_fwd_noalloc(x, U_up, V_up, U_down, V_down, flags: int = 0, out: dict | None = None) -> dict:
    """elas_lowrank_ffn_fwd without a workspace: the library's static device
    scratch is used instead, and nothing is allocated by the call (the output
    tensors must be passed in ``out`` for that; when ``out`` is None they are
    allocated here, by torch, before the call).  Returns the outputs dict."""
    T, d = x.shape
    ab = bool(flags & ELAS_FACTORS_AB)
    r = U_up.shape[0] if ab else U_up.shape[1]
    F = V_up.shape[0] if ab else V_up.shape[1]
    dev = x.device
    dense = bool(flags & ELAS_MODE_DENSE)
    for t, shp, name in ((U_up, (d, r), "U_up"), (V_up, (r, F), "V_up"), (U_down, (F, r), "U_down"),
                         (V_down, (r, d), "V_down")):
        _shape(t, shp[::-1] if ab else shp, name)
    if out is None:
        out = {
            "y": torch.empty((T, d), dtype=torch.bfloat16, device=dev),
            "P": torch.empty((T, r), dtype=torch.bfloat16, device=dev),
            "s_vals": torch.empty((T, F if dense else elas_vals_ld(F)), dtype=torch.bfloat16, device=dev),
            "s_meta": None if dense else torch.empty((T, elas_meta_ld(F)), dtype=torch.uint8, device=dev),
            "Z": torch.empty((T, r), dtype=torch.bfloat16, device=dev),
        }
    _saved_shapes(out, T, d, F, r, dense, with_y=True)
    bf = torch.bfloat16
    _check(lib().elas_lowrank_ffn_fwd_noalloc(
        _ptr(x, bf, "x"), _ptr(U_up, bf, "U_up"), _ptr(V_up, bf, "V_up"), _ptr(U_down, bf, "U_down"),
        _ptr(V_down, bf, "V_down"), T, d, F, r, flags,
        _ptr(out["y"], bf, "y"), _ptr(out["P"], bf, "P"), _ptr(out["s_vals"], bf, "s_vals"),
        _ptr(out["s_meta"], torch.uint8, "s_meta"), _ptr(out["Z"], bf, "Z"), _stream(dev)))
    return out


def elas_lowrank_ffn_bwd(dy, x, U_up, V_up, U_down, V_down, saved: dict, flags: int = 0,
                         grads: dict | None = None, workspace: torch.Tensor | None = None) -> dict:
    """Backward of the low-rank 2:4 FFN given the forward's saved tensors
    (P, s_vals, s_meta, Z).  Returns dict(dx, dU_up, dV_up, dU_down, dV_down).

    flags: 0 (masked derivative), ELAS_BWD_STE (Eq. 4 straight-through) or
    ELAS_MODE_DENSE (after a dense forward)."""
    T, d = x.shape
    r = U_up.shape[1]
    F = V_up.shape[1]
    dev = x.device
    for t, shp, name in ((dy, (T, d), "dy"), (U_up, (d, r), "U_up"), (V_up, (r, F), "V_up"),
                         (U_down, (F, r), "U_down"), (V_down, (r, d), "V_down")):
        _shape(t, shp, name)
    _saved_shapes(saved, T, d, F, r, bool(flags & ELAS_MODE_DENSE), with_y=False)
    if grads is None:
        f32 = torch.float32
        grads = {
            "dx": torch.empty((T, d), dtype=torch.bfloat16, device=dev),
            "dU_up": torch.empty((d, r), dtype=f32, device=dev),
            "dV_up": torch.empty((r, F), dtype=f32, device=dev),
            "dU_down": torch.empty((F, r), dtype=f32, device=dev),
            "dV_down": torch.empty((r, d), dtype=f32, device=dev),
        }
    for k, shp in (("dx", (T, d)), ("dU_up", (d, r)), ("dV_up", (r, F)), ("dU_down", (F, r)), ("dV_down", (r, d))):
        _shape(grads.get(k), shp, k)
    need = elas_lowrank_ffn_bwd_workspace_bytes(T, d, F, r, flags)
    if workspace is None:
        workspace = _workspace(need, dev)
    bf, f32 = torch.bfloat16, torch.float32
    _check(lib().elas_lowrank_ffn_bwd(
        _ptr(dy, bf, "dy"), _ptr(x, bf, "x"), _ptr(U_up, bf, "U_up"), _ptr(V_up, bf, "V_up"),
        _ptr(U_down, bf, "U_down"), _ptr(V_down, bf, "V_down"), T, d, F, r, flags,
        _ptr(saved["P"], bf, "P"), _ptr(saved["s_vals"], bf, "s_vals"),
        _ptr(saved["s_meta"], torch.uint8, "s_meta"), _ptr(saved["Z"], bf, "Z"),
        _ptr(grads["dx"], bf, "dx"), _ptr(grads["dU_up"], f32, "dU_up"), _ptr(grads["dV_up"], f32, "dV_up"),
        _ptr(grads["dU_down"], f32, "dU_down"), _ptr(grads["dV_down"], f32, "dV_down"),
        _ptr(workspace, torch.uint8, "workspace"), 0 if workspace is None else workspace.numel(),
        _stream(dev)))
    return grads


def elas_fullrank_ffn_fwd(x, W_up, W_down, out: dict | None = None) -> dict:
    """Forward of the full-rank ReLU^2 FFN y = relu(x W_up^T)^2 W_down^T with
    W_up [d_ff, d] and W_down [d, d_ff].  Returns dict(y, S), S being the
    dense [T, d_ff] activation."""
    T, d = x.shape
    F = W_up.shape[0]
    dev = x.device
    _shape(W_up, (F, d), "W_up")
    _shape(W_down, (d, F), "W_down")
    if out is None:
        out = {"y": torch.empty((T, d), dtype=torch.bfloat16, device=dev),
               "S": torch.empty((T, F), dtype=torch.bfloat16, device=dev)}
    _shape(out.get("y"), (T, d), "y")
    _shape(out.get("S"), (T, F), "S")
    bf = torch.bfloat16
    _check(lib().elas_fullrank_ffn_fwd(
        _ptr(x, bf, "x"), _ptr(W_up, bf, "W_up"), _ptr(W_down, bf, "W_down"), T, d, F,
        _ptr(out["y"], bf, "y"), _ptr(out["S"], bf, "S"), _stream(dev)))
    return out


def _host_array(a, dtype, shape, name):
    """A C-contiguous host numpy array of ``dtype`` and ``shape`` from a numpy
    array or a (host or device) torch tensor of the same element size."""
    import numpy as np
    if isinstance(a, torch.Tensor):
        a = a.detach().contiguous().cpu().numpy()
    a = np.ascontiguousarray(a)
    if a.dtype.itemsize != np.dtype(dtype).itemsize:
        raise ValueError(f"{name} must have {np.dtype(dtype).itemsize}-byte elements")
    a = a.view(dtype)
    if a.shape != tuple(shape):
        raise ValueError(f"{name} has shape {a.shape}, expected {tuple(shape)}")
    return a


def elas_meta_to_canonical(meta_tiled, M: int, N: int):
    """Canonical metadata [M, N/8] (uint8 numpy) of a compressed S saved by
    elas_lowrank_ffn_fwd in the tiled layout ([M, elas_meta_ld(N)] bytes;
    numpy or torch, copied to the host)."""
    import numpy as np
    src = _host_array(meta_tiled, np.uint8, (M, elas_meta_ld(N)), "meta_tiled")
    out = np.empty((M, N // 8), dtype=np.uint8)
    _check(lib().elas_meta_to_canonical(src.ctypes.data_as(_p), M, N, out.ctypes.data_as(_p)))
    return out


def elas_vals_to_canonical(vals_tiled, M: int, N: int):
    """Canonical kept values [M, N/2] (bf16 bits as uint16 numpy) of a
    compressed S saved by elas_lowrank_ffn_fwd in the tiled layout
    ([M, elas_vals_ld(N)] bf16; numpy or torch, copied to the host)."""
    import numpy as np
    src = _host_array(vals_tiled, np.uint16, (M, elas_vals_ld(N)), "vals_tiled")
    out = np.empty((M, N // 2), dtype=np.uint16)
    _check(lib().elas_vals_to_canonical(src.ctypes.data_as(_p), M, N, out.ctypes.data_as(_p)))
    return out


def elas_debug_sync(enable: bool | None = None) -> bool:
    """Switch the ELAS_DEBUG_SYNC mode (synchronise after every kernel and
    report failures by kernel) on or off; None leaves it.  Returns the
    previous state."""
    return bool(lib().elas_debug_sync(-1 if enable is None else (1 if enable else 0)))


def elas_timing_enable(enable: bool = True) -> None:
    """Start (clearing earlier records) or stop per-kernel event timing."""
    _check(lib().elas_timing_enable(1 if enable else 0))


def elas_timing_only(tag: str | None = None) -> None:
    """Record only the launches of kernel ``tag`` (None: every launch)."""
    _check(lib().elas_timing_only(tag.encode() if tag else None))


def elas_timing_collect() -> dict:
    """{kernel tag: (launches, total ms)} of the launches recorded so far."""
    L = lib()
    n = L.elas_timing_collect()
    if n < 0:
        _check(-n)
    out = {}
    buf = ctypes.create_string_buffer(128)
    for i in range(n):
        launches = _i64()
        ms = ctypes.c_double()
        _check(L.elas_timing_entry(i, buf, 128, ctypes.byref(launches), ctypes.byref(ms)))
        out[buf.value.decode()] = (launches.value, ms.value)
    return out
