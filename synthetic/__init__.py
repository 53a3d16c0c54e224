"""Seeded synthetic inputs for the ELAS low-rank 2:4 FFN.

This module only draws random numbers; it holds none of the method's
arithmetic.  Both the CPU oracle's callers and the GPU path's callers take
their inputs from here, as raw bf16 bit patterns (numpy ``uint16``).

Shapes follow the paper's LLaMA FFN sizes (Table 6 for hidden / intermediate
sizes, Table 1 for the rank r of each model size).  The paper trains on C4,
which is not used here: Gaussian inputs with the fan-in scaled variances below
stand in for the real activations and trained weights.

* x ~ N(0, 1), U_up ~ N(0, 1/d), V_up ~ N(0, 1/r), U_down ~ N(0, 1/d_ff_true),
  V_down ~ N(0, 1/r), dY ~ N(0, 1).  With these scales P = x U_up and
  H = P V_up are about N(0, 1), so roughly half of H is <= 0, which is the
  early-training ReLU^2 sparsity the paper reports in its warm-up ablation.
* When d_ff is padded up to a multiple of 8 (5461 -> 5464 for the 1B shape),
  the pad columns of V_up and the pad rows of U_down are zero.

Values are drawn as float32 from numpy's PCG64 and converted to bf16 by
dropping the low 16 bits (round toward zero).  Truncation is used on purpose:
it needs no rounding arithmetic, so no conversion code is shared with either
side.  Every tensor has its own seed, ``1000 * seed_base + k``.
"""
from __future__ import annotations

import numpy as np

# name -> (T, d, d_ff (padded), d_ff_true, r)
CONFIGS = {
    "llama60m": dict(T=2048, d=512, d_ff=1376, d_ff_true=1376, r=128),
    "llama130m": dict(T=65536, d=768, d_ff=2048, d_ff_true=2048, r=256),
    "llama350m": dict(T=65536, d=1024, d_ff=2736, d_ff_true=2736, r=256),
    "llama1b": dict(T=65536, d=2048, d_ff=5464, d_ff_true=5461, r=512),
    "llama1b_t262144": dict(T=262144, d=2048, d_ff=5464, d_ff_true=5461, r=512),
}

# standalone sparsify workload: h [65536 x 2736] ~ N(0, 1) (350M shape)
SPARSIFY_SHAPE = (65536, 2736)


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def normal_bf16(shape, sigma: float, seed: int, mu: float = 0.0) -> np.ndarray:
    """N(mu, sigma^2) samples as bf16 bit patterns (float32 truncated)."""
    g = _rng(seed)
    v = g.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        v *= np.float32(sigma)
    if mu != 0.0:
        v += np.float32(mu)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def ffn_inputs(T: int, d: int, d_ff: int, r: int, d_ff_true: int | None = None,
               seed_base: int = 0) -> dict:
    """All inputs of one FFN forward + backward, as bf16 bits.

    Keys: x [T,d], U_up [d,r], V_up [r,d_ff], U_down [d_ff,r], V_down [r,d],
    dY [T,d].
    """
    if d_ff_true is None:
        d_ff_true = d_ff
    s = 1000 * seed_base
    out = {
        "x": normal_bf16((T, d), 1.0, s + 1),
        "U_up": normal_bf16((d, r), 1.0 / np.sqrt(d), s + 2),
        "V_up": normal_bf16((r, d_ff), 1.0 / np.sqrt(r), s + 3),
        "U_down": normal_bf16((d_ff, r), 1.0 / np.sqrt(d_ff_true), s + 4),
        "V_down": normal_bf16((r, d), 1.0 / np.sqrt(r), s + 5),
        "dY": normal_bf16((T, d), 1.0, s + 6),
    }
    if d_ff_true < d_ff:
        out["V_up"][:, d_ff_true:] = 0
        out["U_down"][d_ff_true:, :] = 0
    return out


def exact_p_inputs(T: int, d: int, d_ff: int, r: int, d_ff_true: int | None = None,
                   seed_base: int = 0) -> dict:
    """Like ffn_inputs, but x and U_up are drawn on coarse grids so that
    every sum of x U_up is exact in binary32 (and float64): x ~ N(0, 1) on
    multiples of 1/8 in [-4, 4] (at most 6 significant bits), U_up ~ N(0, 1/d)
    on multiples of 2^-g, g = floor(log2(64 sqrt(d))), at most 255 grid steps
    (8 bits).  Both are exact bf16 values, so every implementation that
    accumulates in binary32 holds the same P, and differences downstream come
    from the later products only.  The other tensors are those of
    ffn_inputs."""
    out = ffn_inputs(T, d, d_ff, r, d_ff_true, seed_base)
    s = 1000 * seed_base
    g = _rng(s + 7)
    x = np.clip(np.rint(g.standard_normal((T, d)) * 8.0), -32, 32) / 8.0
    step = 2.0 ** -int(np.floor(np.log2(64.0 * np.sqrt(d))))
    u = np.clip(np.rint(g.standard_normal((d, r)) / np.sqrt(d) / step), -255, 255) * step
    out["x"] = (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    out["U_up"] = (u.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return out


def fullrank_inputs(T: int, d: int, d_ff: int, d_ff_true: int | None = None, seed_base: int = 0) -> dict:
    """Inputs of the full-rank ReLU^2 FFN forward, as bf16 bits.

    Keys: x [T,d] ~ N(0,1); W_up [d_ff,d] ~ N(0,1/d), so that the
    pre-activation is about N(0,1) as in the low-rank block; W_down [d,d_ff]
    ~ N(0,1/d_ff_true).  Weights are in the orientation of a linear layer
    (output features as rows).  Pad rows of W_up and pad columns of W_down
    (feature index >= d_ff_true) are zero.
    """
    if d_ff_true is None:
        d_ff_true = d_ff
    s = 1000 * seed_base + 500
    out = {
        "x": normal_bf16((T, d), 1.0, s + 1),
        "W_up": normal_bf16((d_ff, d), 1.0 / np.sqrt(d), s + 2),
        "W_down": normal_bf16((d, d_ff), 1.0 / np.sqrt(d_ff_true), s + 3),
    }
    if d_ff_true < d_ff:
        out["W_up"][d_ff_true:, :] = 0
        out["W_down"][:, d_ff_true:] = 0
    return out


def config_inputs(name: str, T: int | None = None, seed_base: int | None = None) -> dict:
    """Inputs of a named workload; ``T`` overrides the token count."""
    c = dict(CONFIGS[name])
    if T is not None:
        c["T"] = T
    if seed_base is None:
        seed_base = list(CONFIGS).index(name)
    return ffn_inputs(c["T"], c["d"], c["d_ff"], c["r"], c["d_ff_true"], seed_base)


def h_input(M: int, N: int, seed: int, mu: float = 0.0, levels: int | None = None) -> np.ndarray:
    """Activation h [M, N] ~ N(mu, 1) as bf16 bits.

    mu = -0.994 and mu = -2.054 give about 84 % and 98 % zeros after ReLU^2,
    the range the paper reports after warm-up.  With ``levels`` the values are
    quantised to that many integers (ties on purpose).
    """
    g = _rng(seed)
    v = g.standard_normal(size=(M, N), dtype=np.float32)
    if mu != 0.0:
        v += np.float32(mu)
    if levels is not None:
        v = np.round(np.clip(v, -2.0, 2.0) * (levels / 4.0)).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def uniform_int_bf16(shape, lo: int, hi: int, seed: int, scale_log2: int = 0) -> np.ndarray:
    """Integers in [lo, hi] times 2**scale_log2, as bf16 bits.

    Small integers times a power of two are exact in bf16 and their sums stay
    exact in fp32 and fp64, so both sides see identical values.
    """
    g = _rng(seed)
    v = g.integers(lo, hi + 1, size=shape).astype(np.float32) * np.float32(2.0 ** scale_log2)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def sparse_sign_bf16(shape, density: float, seed: int, scale_log2: int = 0) -> np.ndarray:
    """+-2**scale_log2 at a random fraction ``density`` of the positions, 0
    elsewhere, as bf16 bits.  Sparse small integers keep every sum of the
    block exact in binary32 even at the largest model shape."""
    g = _rng(seed)
    v = np.where(g.random(shape) < density, g.choice(np.array([-1.0, 1.0]), size=shape), 0.0)
    v = (v * 2.0 ** scale_log2).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)
