"""Plain fp64 CPU oracle for the Allegro channel-wise Clebsch-Gordan tensor product.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.  The
GPU product path (``paper_2504_16068_amd``) never imports it, and this package
never imports the product path: the two share no code, tables or constants.

What it computes (arxiv 2504.16068, §II.D "Optimized Tensor Product Kernel"):
the per-edge, channel-wise tensor product that the paper names the most
expensive operation of the Allegro architecture, forward and first derivative
(the VJP that inference-time forces need), together with the environment
embedding it consumes.  The paper defers the formula to the Allegro papers it
cites; the operation is restated in ``tp.py``.  Precision follows the paper's
Appendix "Mixed-Precision Architecture": the tensor product runs in fp32 on
the GPU, and this oracle evaluates the exact definition in fp64 on the very
same fp32 input values.

Modules
  irreps  -- irreducible-representation lists and the allowed (l1,l2 -> l3) paths
  cg      -- complex Clebsch-Gordan coefficients by Racah's formula (exact
             rationals), the complex-to-real change of basis, and the
             normalisation / sign rule of the real coupling tensors
  sh      -- real spherical harmonics (associated-Legendre recurrence + the
             same change of basis), component normalisation
  wigner  -- Wigner-D matrices of the real basis, fitted from the harmonics
             (a test tool for equivariance)
  tp      -- environment embedding, tensor product forward and backward, each
             in a nested-loop form and a per-path einsum form

Every function whose result has no independent pin says "parity unpinned" in
its docstring.  The only such items are conventions (basis signs, the sign
rule of each coupling tensor, the normalisation of the harmonics), which every
invariant holds for under any consistent choice.
"""
