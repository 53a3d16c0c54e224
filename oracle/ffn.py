"""The ELAS low-rank ReLU^2 FFN with 2:4 activation sparsity (oracle; tests only).

Block (Fig. 1 caption, Sec. 3): the input goes through the two low-rank
factors of the up projection, then ReLU^2 (Eq. 2), then 2:4 sparsification
(Algorithm 1 / Eq. 3), then the two low-rank factors of the down projection.

Factors (Eq. 1, Sec. 3.1): a linear map W = A B with A [d_out x r] and
B [r x d_in].  Acting on row vectors (tokens as rows) this is x W^T = x B^T A^T;
this implementation names the two right-multiplied factors U = B^T and V = A^T:

    P = x U_up            x [T, d],  U_up [d, r]
    H = P V_up            V_up [r, d_ff]
    s = relu(H)^2         Eq. 2
    S = mask_top2(s) * s  Algorithm 1, Eq. 3 (groups of 4 along d_ff)
    Z = S U_down          U_down [d_ff, r]
    Y = Z V_down          V_down [r, d]

Backward (Sec. 3.3.2, Sec. 3.4: plain backpropagation through the low-rank
factors; the sparsification is the only non-differentiable step):

    dZ = dY V_down^T,  dV_down = Z^T dY
    dS = dZ U_down^T,  dU_down = S^T dZ
    dH = dS * mask * 2 relu(H)       (default: derivative of the sparsified
                                      forward; the mask is held fixed)
    dH = dS * 2 relu(H)              (ste=True: Eq. 4 literally, sparsify
                                      treated as the identity)
    dP = dH V_up^T,    dV_up = P^T dH
    dx = dP U_up^T,    dU_up = x^T dP

All arithmetic is float64 (matrix products by numpy).  With ``bf16io=True``
the tensors the GPU path stores in bf16 (P, H before ReLU^2, the kept values
of S, Z, Y, dZ, dH, dP, dx) are rounded to bf16 (nearest, ties to even) at the
same points; weight gradients are never rounded.  The default masked backward
and the bf16 rounding points are readings of the paper; see the module
docstring of ``oracle`` for what pins them.
"""
from __future__ import annotations

import numpy as np

from . import bf16
from .sparsify import relu2, top2_mask


def _rounder(bf16io: bool):
    return bf16.round_f64 if bf16io else (lambda a: a)


def forward(x, U_up, V_up, U_down, V_down, *, bf16io: bool = True, sparse: bool = True, mask=None):
    """Forward pass.  Inputs are float64 arrays (exact bf16 values).

    Returns a dict with Y and the intermediates P, H, s, mask, S, Z.
    ``sparse=False`` skips Algorithm 1 (dense activations, the paper's
    warm-up phase).  ``mask`` (boolean, H's shape) replaces Algorithm 1's
    selection by a given one, e.g. the selection of the bf16-rounded block
    applied to the plain float64 block, so that the two differ only in
    their arithmetic.
    """
    rb = _rounder(bf16io)
    P = rb(x @ U_up)
    H = rb(P @ V_up)
    s = relu2(H)
    if mask is None:
        mask = top2_mask(s) if sparse else np.ones(s.shape, dtype=bool)
    S = rb(np.where(mask, s, 0.0))
    Z = rb(S @ U_down)
    Y = rb(Z @ V_down)
    return {"Y": Y, "P": P, "H": H, "s": s, "mask": mask, "S": S, "Z": Z}


def backward(dY, x, U_up, V_up, U_down, V_down, fwd, *, bf16io: bool = True,
             ste: bool = False):
    """Backward pass given the forward's dict; returns all gradients."""
    rb = _rounder(bf16io)
    P, H, mask, S, Z = fwd["P"], fwd["H"], fwd["mask"], fwd["S"], fwd["Z"]
    dZ = rb(dY @ V_down.T)
    dV_down = Z.T @ dY
    dS = dZ @ U_down.T
    dU_down = S.T @ dZ
    g = dS * 2.0 * np.where(H > 0, H, 0.0)
    dH = rb(g if ste else np.where(mask, g, 0.0))
    dP = rb(dH @ V_up.T)
    dV_up = P.T @ dH
    dU_up = x.T @ dP
    dx = rb(dP @ U_up.T)
    return {"dx": dx, "dU_up": dU_up, "dV_up": dV_up, "dU_down": dU_down,
            "dV_down": dV_down, "dZ": dZ, "dS": dS, "dH": dH, "dP": dP}


def fullrank_forward(x, W_up, W_down, *, bf16io: bool = True):
    """Forward of the full-rank ReLU^2 FFN that Table 3 (Sec. 4.2.3) compares
    ELAS against.  W_up [d_ff, d] and W_down [d, d_ff] are the full matrices
    W of Eq. 1 (acting on column vectors); with tokens as rows:
    H = x W_up^T, S = relu(H)^2, Y = S W_down^T.  With ``bf16io`` H (before
    ReLU^2), S and Y are rounded to bf16, the same points as the low-rank
    block's H, S and Y.  Returns dict(Y, H, S)."""
    rb = _rounder(bf16io)
    H = rb(x @ W_up.T)
    S = rb(relu2(H))
    Y = rb(S @ W_down.T)
    return {"Y": Y, "H": H, "S": S}


def from_bits(inputs: dict) -> dict:
    """bf16 bit arrays -> exact float64 arrays (same keys)."""
    return {k: bf16.to_f64(v) for k, v in inputs.items()}


def run(inputs_bits: dict, *, bf16io: bool = True, ste: bool = False, sparse: bool = True, mask=None):
    """Forward + backward on a dict of bf16 bit arrays (x, U_up, V_up, U_down,
    V_down, dY).  Returns (forward dict, backward dict)."""
    a = from_bits(inputs_bits)
    f = forward(a["x"], a["U_up"], a["V_up"], a["U_down"], a["V_down"],
                bf16io=bf16io, sparse=sparse, mask=mask)
    b = backward(a["dY"], a["x"], a["U_up"], a["V_up"], a["U_down"], a["V_down"], f,
                 bf16io=bf16io, ste=ste)
    return f, b
