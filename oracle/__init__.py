"""CPU oracle for the DS-MPNN hot path (arXiv 2402.15106).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
CPU implementation of what the GPU path computes.  Only the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
product path (the HIP library and its Python binding) never does, and the two
share no code.

Contents, each following the paper passage named in its module docstring:

* ``rng``          -- SplitMix64, the counter-based generator both sides use
                      for every random draw the method makes.
* ``sampling``     -- Nystrom node sampling (Sec. 2.1; Algorithm 1, node
                      sampling step).
* ``radius_graph`` -- radius-graph kernel construction with the edge cap
                      (Sec. 2.1; Algorithm 1, edge-index creation and edge
                      sampling steps).
* ``nnconv``       -- edge attributes, the edge-conditioned convolution of
                      eq. (1) / eq. (ii) with root term and residual hop
                      update (Algorithm 1, graph-convolution step), and its
                      hand-derived backward pass.
* ``hop``          -- encoder / decoder perceptrons, the masked MSE and the
                      hop loop of Algorithm 1 (eqs. (i)-(iv)) on one
                      sub-domain, forward and backward.
* ``infer``        -- sub-domain inference with reassembly (Sec. 3, testing
                      procedure).

Floating point: the layer runs in float64.  The radius test runs in float32
in a fixed evaluation order (no fused multiply-add), because the paper fixes
no precision and the GPU must reproduce the edge set bit for bit.
"""

from . import rng, sampling, radius_graph, nnconv, hop, infer  # noqa: F401
