"""CPU oracle for the ELAS low-rank 2:4-sparse FFN block.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import or call anything here.
The product path (the HIP library and its Python binding) never does, and
this package imports nothing from it.

The oracle is a plain, slow restatement of the paper (ELAS, arXiv 2605.03667):

* ``oracle.bf16``     -- bf16 round-to-nearest-even from float64, by definition.
* ``oracle.sparsify`` -- Eq. 2 (ReLU^2), Algorithm 1 / Eq. 3 (2:4 top-2 of
                         each group of 4 along the feature dimension) and the
                         compressed storage (values + 2-bit indices, Sec. 4.2.2).
* ``oracle.ffn``      -- the low-rank FFN of Fig. 1 built from Eq. 1 factors,
                         forward, and backward with the masked gradient
                         (default) or the literal straight-through estimator of
                         Eq. 4; ``fullrank_forward`` is the full-rank ReLU^2
                         FFN that Table 3 compares against.

Arithmetic is float64 throughout.  Optionally (``bf16io=True``) values are
rounded to bf16 at the points where the GPU path stores bf16 tensors; the
paper trains in BF16 (Sec. 4.1, Model Architecture) and these rounding points
are this implementation's reading of that.

Pins (tests marked ``not gpu``): brute-force enumeration of the six keep
patterns, exact bf16 rounding against rational arithmetic and torch's
conversion, finite differences of the full forward, torch autograd on cases
that reduce to a dense FFN, closed-form special cases, the storage ratio
of Table 2, and for the full-rank block explicit loops, the factorised-weight
identity with the low-rank block and its 2-homogeneity.  Nothing here is "parity unpinned" except the padding reading for
d_ff = 5461 (the paper does not say how it handles a width that is not a
multiple of 4).
"""
