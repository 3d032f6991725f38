"""Float64 CPU oracle for the MatRIS-MoE training step (TEST INFRASTRUCTURE).

This package is the plain, slow reference that the HIP path is checked
against.  Only the test-suite, the package smoke check and the CPU-baseline
leg of the benchmark may import it; the product path never calls it and has
no CPU fallback.  It shares no code with the HIP path: it imports nothing
from the product package, and it takes the seeded synthetic arrays as plain
NumPy inputs.

What it computes (paper Sec. "MatRIS" and Sec. "Algorithmic innovation",
together with the model reading written out in the module docstrings):

* ``neighbors``  -- periodic neighbour list under the pinned float32 test,
                    canonical (i, j, n) order, reverse-edge map, triplets.
* ``basis``      -- Bessel radial basis with polynomial envelope, SiLU
                    family, Legendre polynomials; closed-form derivatives.
* ``model``      -- energy, conservative forces F = -dE/dR, the
                    energy+force loss, and every weight gradient of the
                    loss (second order), hand-derived.
* ``threebody``  -- bond-triplet features (Legendre of the bond angle times a
                    radial basis), their tangents and displacement adjoints.

Every function cites the passage of the paper it follows.  Where the paper
is silent the reading used is stated in the docstring.
"""

from .neighbors import neighbor_list, reverse_map, triplet_list, image_range
from .basis import bessel_basis, envelope, silu, silu_d1, silu_d2, legendre
from .model import (Params, route, forward_energy, forces, loss_and_seeds,
                    weight_gradient, training_step, energy_tangent)

__all__ = [
    "neighbor_list", "reverse_map", "triplet_list", "image_range",
    "bessel_basis", "envelope", "silu", "silu_d1", "silu_d2", "legendre",
    "Params", "route", "forward_energy", "forces", "loss_and_seeds",
    "weight_gradient", "training_step", "energy_tangent",
]
