"""ReLU^2 and 2:4 activation sparsification (oracle; tests only).

Follows ELAS (arXiv 2605.03667):

* Eq. 2 (Sec. 3.2): ReLU^2(z) = max(0, z)^2.
* Algorithm 1 and Eq. 3 (Sec. 3.3.1): each row of the activation z [M x N] is
  cut into consecutive groups of 4 along the feature dimension; inside a group
  the 2 entries of largest absolute value are kept and the other 2 are set to
  zero; sparsify(z) = mask_top2(z) * z.
* Sec. 4.2.2: the sparse activation is stored as its kept values plus compact
  index information.

Readings where the paper is silent:

* Exactly 2 slots are kept per group, even when fewer than 2 entries are
  nonzero (a kept slot may hold 0).  The paper's definition of 2:4 says "at
  least 2 zeros"; Algorithm 1 keeps the top 2.
* Ties in |z| go to the lower index (a stable sort).
* relu(NaN) is 0 (the comparison "z > 0" is false for NaN).

Compressed layout (the build's own encoding, canonical form): for row i and
group j (features 4j..4j+3), ``vals[i, 2j]`` and ``vals[i, 2j+1]`` hold the
two kept values in ascending feature order, and the group's 4-bit code
``i0 | (i1 << 2)`` (i0 < i1, the kept positions inside the group) sits in byte
``meta[i, j // 2]``, low nibble for even j, high nibble for odd j.
"""
from __future__ import annotations

import numpy as np

from . import bf16


def relu2(z: np.ndarray) -> np.ndarray:
    """Eq. 2: (max(0, z))^2, with relu(NaN) = 0."""
    r = np.where(z > 0, z, 0.0)
    return r * r


def top2_mask(z: np.ndarray) -> np.ndarray:
    """Algorithm 1's mask: per row, per group of 4, keep the 2 largest |z|.

    Returns a boolean array of z's shape.  The group's absolute values are
    ordered by a stable sort on decreasing magnitude, so among equal magnitudes
    the lower index comes first; the first two positions of that order are kept.
    """
    M, N = z.shape
    if N % 4:
        raise ValueError("the feature dimension must be a multiple of 4")
    groups = z.reshape(M, N // 4, 4)
    abs_group = np.abs(groups)
    order = np.argsort(-abs_group, axis=-1, kind="stable")
    keep = np.zeros(groups.shape, dtype=bool)
    np.put_along_axis(keep, order[..., :2], True, axis=-1)
    return keep.reshape(M, N)


def sparsify24(z: np.ndarray) -> np.ndarray:
    """Eq. 3: mask_top2(z) * z (dense result)."""
    return np.where(top2_mask(z), z, 0.0)


def compress(values: np.ndarray, mask: np.ndarray):
    """Kept values and 2-bit indices of a 2:4 masked matrix (canonical layout).

    ``values`` is any array of the matrix's shape (its entries at the kept
    positions are taken); ``mask`` must keep exactly 2 of every 4.  Returns
    (vals [M, N/2] of values' dtype, meta [M, N/8] uint8).
    """
    M, N = mask.shape
    if N % 8:
        raise ValueError("the feature dimension must be a multiple of 8")
    km = mask.reshape(M, N // 4, 4)
    if not np.all(km.sum(axis=-1) == 2):
        raise ValueError("mask does not keep exactly 2 of every 4")
    pos = np.nonzero(km)[2].reshape(M, N // 4, 2)      # row-major: i0 < i1
    vals = np.take_along_axis(values.reshape(M, N // 4, 4), pos, axis=-1).reshape(M, N // 2)
    code = (pos[..., 0] | (pos[..., 1] << 2)).astype(np.uint8)   # [M, N/4]
    meta = (code[:, 0::2] | (code[:, 1::2] << 4)).astype(np.uint8)
    return vals, meta


def decompress(vals: np.ndarray, meta: np.ndarray, N: int, fill=0):
    """Dense [M, N] matrix and boolean mask from (vals, meta)."""
    M = meta.shape[0]
    code = np.empty((M, N // 4), dtype=np.uint8)
    code[:, 0::2] = meta & 0xF
    code[:, 1::2] = meta >> 4
    i0 = code & 3
    i1 = code >> 2
    dense = np.full((M, N // 4, 4), fill, dtype=vals.dtype)
    v = vals.reshape(M, N // 4, 2)
    np.put_along_axis(dense, i0[..., None].astype(np.int64), v[..., :1], axis=-1)
    np.put_along_axis(dense, i1[..., None].astype(np.int64), v[..., 1:], axis=-1)
    mask = np.zeros((M, N // 4, 4), dtype=bool)
    np.put_along_axis(mask, i0[..., None].astype(np.int64), True, axis=-1)
    np.put_along_axis(mask, i1[..., None].astype(np.int64), True, axis=-1)
    return dense.reshape(M, N), mask.reshape(M, N)


RELU2 = 0   # s = relu(h)^2, then Algorithm 1 on s  (the ELAS activation)
RAW = 1     # Algorithm 1 directly on z (signed values kept)


def sparsify24_bf16(h_bits: np.ndarray, mode: int = RELU2):
    """The standalone sparsify contract on a bf16 activation.

    RELU2: s = relu(h)^2 (exact in float64 for every bf16 h), Algorithm 1 on s,
           kept values rounded to bf16 (nearest, ties to even).
    RAW:   Algorithm 1 on z = h itself; kept values are h unchanged.
    Returns (vals bits [M, N/2] uint16, meta [M, N/8] uint8).
    """
    h = bf16.to_f64(h_bits)
    if mode == RELU2:
        s = relu2(h)
        mask = top2_mask(s)
        vals, meta = compress(bf16.from_f64(s), mask)
    elif mode == RAW:
        mask = top2_mask(h)
        vals, meta = compress(np.asarray(h_bits, dtype=np.uint16), mask)
    else:
        raise ValueError("unknown mode")
    return vals.astype(np.uint16), meta
