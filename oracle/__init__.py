"""fp64 CPU oracle for the channelwise Clebsch-Gordan message-passing convolution.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: only the test-suite, the package smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP library
(no tables, no helpers); the one module both sides read is the seeded input
generator package ``synth``, which holds none of the method's arithmetic.

Everything here is the plain definition, written out in float64:

* ``irreps``  -- irreps strings and the path list (paper App. A.3, the
  "Tensor product" item; App. E.1 "Mathematical operations" for the map i3).
* ``cg``      -- complex Clebsch-Gordan coefficients from Racah's closed
  formula, the complex-to-real change of basis fitted on sample points, and
  the real coupling tensors with the canonical sign rule.
* ``sh``      -- real spherical harmonics from the textbook Cartesian
  (solid-harmonic) formula, component normalisation, and their Jacobian by
  float64 autograd.
* ``wigner``  -- Wigner-D matrices by least squares (tests only).
* ``tp``      -- the weighted tensor product, eq. (tensor_product_formula) and
  eq. (edge_scalar_weighting) of App. E.1.
* ``conv``    -- the message-passing convolution, eq.
  (message_passing_convolution), and its cotangents, eq. (conv-bwd).
* ``graph``   -- receiver/sender CSR by a stable argsort.

Every function says which passage it follows.  Where the paper leaves a
convention open (normalisation, real-basis phase, axes, path order) the
adopted reading is stated next to the code that applies it.
"""
