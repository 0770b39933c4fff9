"""CPU oracle for the CP tensor-product message-passing layer -- TEST
INFRASTRUCTURE ONLY.

This package is a plain, slow, double-precision restatement of what the layer
computes, written from the paper (arXiv 2507.01131) so that the GPU path can
be checked against it.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import it; the product path never does and
shares no code with it.

Modules
  sh        real spherical (solid) harmonics and their gradient, closed form
  cg        Clebsch-Gordan coefficients (Racah's formula) and the real basis
            (Sec. 2, eq. clebsch_gordan)
  wigner    real Wigner-D matrices (Sec. 3.4 and App. B.1)
  cg_tensor the coefficient tensor M over all paths and the dense tensor
            product (Sec. 3.1, eq. bilinear)
  cp        CP decomposition of M by alternating least squares, the
            universality construction, error metrics (Sec. 3.1 eq. cp,
            Sec. 3.3, Sec. 3.4, Sec. 4.1, App. B)
  layer     the message-passing layer by direct per-edge summation and its
            backward (Sec. 3.1 eq. approximate, Sec. 3.2)
  dense_layer
            the exact CG tensor-product layer path by path, the comparator
            of the CP layer (Sec. 2 eq. clebsch_gordan, Sec. 3.2), with the
            shared channel weight or with one channel weight per path (the
            product without path-weight sharing)
  attention the graph-attention block that consumes the CP messages (one
            reading of Sec. 4.1 "Model Design": MLP attention logits from
            invariant edge inputs, a softmax over each destination's edges
            per head, the heads weighting channel blocks of the messages)
  radius_graph
            the edges the layer consumes: every atom pair of a system (and
            its periodic images) closer than the cutoff, with an optional
            nearest-neighbour cap, by brute force in float32 (App. "Model and
            Training Configurations")

Parity status: every function is pinned by the tests in tests/test_oracle_*.py
against closed forms, library routines, invariants or brute force, except the
fitted CP factor values themselves, which are not unique (any local optimum
of the fit is acceptable) -- parity unpinned for those values; what is pinned
is the fit's error behaviour and the exact construction of Thm. 2.
"""
