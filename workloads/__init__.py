"""Seeded synthetic workloads shared by the tests, the smoke check and the benchmark.

This module synthesises INPUTS only: candidate point sets shaped like the
paper's meshes, node features, latent node features, layer parameters and
upstream gradients.  It performs none of the method's arithmetic (no
sampling, no neighbour search, no message passing); both the GPU path and the
CPU oracle consume what it produces.

The paper's datasets (Darcy flow on a 421x421 grid, the AirfRANS airfoil
meshes, the 3-D backward-facing step; Sec. 4) are not available, so these
generators stand in for them with the same shapes, sizes and structure:

  1  2-D unit square, 64x64 grid, 1,024 sampled, features (x, y, a) with a a
     log-normal random field of length scale 0.1; d = 32, MLP 6->64->64, 2
     layers, float32, r = 0.08, no cap.
  2  the same field on a 256x256 grid, 8,192 sampled, r = 0.04; d = 64, MLP
     6->128->128, 4 layers, bf16 operands.
  3  airfoil-like 2-D mesh: candidates with density ~ 1/(0.01 + distance to a
     NACA-0012 outline) in [-2,3]x[-1.5,1.5] minus the airfoil; 32,768
     sampled, features (x, y, wall distance, u_inf, v_inf); r = 0.05, kNN cap
     32; d = 64, 6 layers, bf16.
  4  3-D channel [0,10]x[0,1]^2 minus the step x<1, z<0.5: a 0.02 lattice
     keeping every point within 0.1 of a wall and a seeded quarter of the
     rest (4x refinement near walls); 100,000 sampled, features (x, y, z,
     wall distance); r = 0.06, kNN cap 24; d = 64, MLP 8->128->128, 4 layers,
     bf16.
  5  one GPU's share of a slab decomposition of case 4: owned slab
     2.5 <= x <= 5.0 (262,144 sampled nodes) plus halo strips 2r wide on both
     sides sampled at the same rate, from a 0.0125 lattice; d = 128, MLP
     8->256->256, 4 layers, bf16.

Seeds: geometry and features 1000+k, parameters 2000+k, upstream gradient
3000+k, the sampler seed handed to the library 4000+k; numpy PCG64.
"""

from .configs import Workload, make_config, bf16_round, layer_params, hop_setup, subdomain_boxes, CONFIG_IDS  # noqa: F401
