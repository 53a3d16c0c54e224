"""Shared test utilities: bf16 bit arrays <-> torch tensors, the padded and
tiled compressed layouts, and the comparison protocol between the GPU path
and the oracle.  Holds none of the method's arithmetic."""
from __future__ import annotations

import numpy as np
import torch


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bit array -> bf16 tensor on cuda:0."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda:0")


def host_bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> uint16 bit array on the host."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def vals_ld(N: int) -> int:
    return 32 * ((N + 63) // 64)


def meta_ld(N: int) -> int:
    return 8 * ((N + 63) // 64)


def pad_compressed(vals: np.ndarray, meta: np.ndarray, N: int):
    """Canonical (vals [M, N/2], meta [M, N/8]) -> the library's padded rows:
    padding groups hold zeros and code 0x4 (positions 0 and 1)."""
    M = vals.shape[0]
    v = np.zeros((M, vals_ld(N)), dtype=vals.dtype)
    v[:, : N // 2] = vals
    m = np.full((M, meta_ld(N)), 0x44, dtype=np.uint8)
    m[:, : N // 8] = meta
    return v, m


def untile(a, T: int, ld: int, bw: int):
    """Row-major [T, ld] copy of a compressed tensor in the tiled layout the
    FFN uses for its saved S (include/elas.h): rows in blocks of 256 (the last
    block holds the R remaining rows), each block cut into entry blocks of bw
    (32 values or 8 metadata bytes) that hold R rows x bw entries row-major,
    one after the other.  Works on numpy arrays and torch tensors (on their
    device); only the first T * ld entries are read."""
    is_torch = isinstance(a, torch.Tensor)
    flat = a.reshape(-1)[: T * ld]
    parts = []
    for t0 in range(0, T, 256):
        R = min(256, T - t0)
        blk = flat[t0 * ld: t0 * ld + R * ld].reshape(ld // bw, R, bw)
        blk = blk.permute(1, 0, 2) if is_torch else blk.transpose(1, 0, 2)
        parts.append(blk.reshape(R, ld))
    if not parts:
        return a.reshape(0, ld)
    return torch.cat(parts) if is_torch else np.concatenate(parts)


def tile(a: np.ndarray, bw: int) -> np.ndarray:
    """Inverse of untile for a row-major [T, ld] numpy array (flat result)."""
    T, ld = a.shape
    parts = []
    for t0 in range(0, T, 256):
        R = min(256, T - t0)
        parts.append(a[t0: t0 + R].reshape(R, ld // bw, bw).transpose(1, 0, 2).reshape(-1))
    return np.concatenate(parts) if parts else a.reshape(-1)


def check_padding(vals: np.ndarray, meta: np.ndarray, N: int):
    """The padding of the library's compressed rows holds zeros / code 0x4."""
    assert np.all(vals[:, N // 2:] == 0), "padding values must be zero"
    assert np.all(meta[:, N // 8:] == 0x44), "padding codes must be 0x4"


def rel_fro(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    if nb == 0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / nb)


def mask_gate(gpu_mask: np.ndarray, ref_mask: np.ndarray, ref_keys: np.ndarray, h_range, rel: float = 1e-2):
    """Mask comparison between the GPU's 2:4 selection and the oracle's.

    Every group where the two differ must be the stable top-2 (ties to the
    lower index) of some h that the binary32 accumulation of the up
    projection can produce: ``h_range(rows, cols)`` returns the smallest and
    largest possible bf16 h (oracle.bounds.h_range) for those token rows and
    feature columns.  With each element the GPU keeps at its largest
    possible relu(h) and each one it drops at its smallest (the key ReLU^2
    orders like relu(h)), every kept key must exceed every dropped key, or
    equal it at a lower index.  Groups for which no such h exists are
    "unexplained".

    Also counted (the window the tolerance of the comparison names): groups
    where an entry kept only by the GPU and one kept only by the oracle have
    oracle keys ``ref_keys`` more than ``rel`` apart relative to the larger.

    Returns dict(groups, flips, outside_rel, unexplained)."""
    M, N = ref_mask.shape
    g = gpu_mask.reshape(M, N // 4, 4)
    o = ref_mask.reshape(M, N // 4, 4)
    k = ref_keys.reshape(M, N // 4, 4)
    idx = np.argwhere(np.any(g != o, axis=-1))
    out = {"groups": M * N // 4, "flips": int(len(idx)), "outside_rel": 0, "unexplained": 0}
    if len(idx) == 0:
        return out
    rows = np.unique(idx[:, 0])
    cols = np.unique((idx[:, 1][:, None] * 4 + np.arange(4)[None, :]).ravel())
    lo, hi = h_range(rows, cols)
    rpos = {int(v): i for i, v in enumerate(rows)}
    cpos = {int(v): i for i, v in enumerate(cols)}
    for i, j in idx:
        ri, ci = rpos[int(i)], [cpos[int(4 * j + q)] for q in range(4)]
        khi, klo = np.maximum(hi[ri, ci], 0.0), np.maximum(lo[ri, ci], 0.0)
        kept, dropped = np.nonzero(g[i, j])[0], np.nonzero(~g[i, j])[0]
        if not all(khi[a] > klo[b] or (khi[a] == klo[b] and a < b) for a in kept for b in dropped):
            out["unexplained"] += 1
        only_gpu, only_ref = np.nonzero(g[i, j] & ~o[i, j])[0], np.nonzero(o[i, j] & ~g[i, j])[0]
        if any(abs(k[i, j, f] - k[i, j, e]) > rel * max(k[i, j, e], k[i, j, f]) for e in only_gpu for f in only_ref):
            out["outside_rel"] += 1
    return out


def s_in_range(gpu_s: np.ndarray, s_lo: np.ndarray, s_hi: np.ndarray) -> bool:
    """Dense activations: every GPU value of s lies in the oracle's range of
    possible values (oracle.bounds.s_range)."""
    return bool(np.all((s_lo <= gpu_s) & (gpu_s <= s_hi)))
