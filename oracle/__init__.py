"""CPU oracle for the small-footprint MLIP energy/force/virial path.

TEST INFRASTRUCTURE ONLY.  Only `tests/`, `__graft_entry__.smoke()` and the
`cpu_baseline` leg of `bench.py` may import or run anything in this package.
The product path (the HIP library and its Python binding) never calls it and
shares no code with it.

The oracle is a plain, slow, float64 NumPy transcription of the method as the
paper defines it (Section 3.1, Eqs. 1-10; Section 3.3 for the angular basis;
Section 4.1 for the network architecture).  Every step is the textbook
definition: no fusion, tiling, recomputation or reassociation.

Modules:
  neighbors  neighbour lists (brute force and a cell list giving the same set)
  angular    Cartesian monomials, the irreducible harmonic projection Q_l
  model      weight-blob unpacking, encoder, descriptor, regression head,
             explicit backward pass (W, U, V, partial forces), virial
  md         velocity-Verlet driver used for trajectory comparisons
"""
from .neighbors import wrap_positions, min_image, brute_force_neighbors, cell_list_neighbors, neighbor_list
from .angular import (monomial_exponents, multinomial_diag, laplacian_matrix, harmonic_projection,
                      angular_basis, angular_features)
from .model import Model, evaluate
from .md import velocity_verlet

__all__ = [
    "wrap_positions", "min_image", "brute_force_neighbors", "cell_list_neighbors", "neighbor_list",
    "monomial_exponents", "multinomial_diag", "laplacian_matrix", "harmonic_projection",
    "angular_basis", "angular_features", "Model", "evaluate", "velocity_verlet",
]
