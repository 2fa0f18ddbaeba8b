"""CPU FP64 oracle for the batched PaiNN screening forward pass.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the GPU library (no kernels, headers, tables or helpers); the two meet only at
the synthetic inputs of the `synth` module.

Contents:
  neighbors.radius_graph   brute-force radius graph of one structure (all
                           image pairs, sorted by receiver, sender, shift)
  neighbors.batch_graph    the same as one CSR over a batch
  painn.structure_forward  FP64 PaiNN energy by the edge-list formulation
  painn.structure_forward_dense  the same by dense masked tensors (tiny inputs)
  painn.batch_energies     per-structure energies of a batch
  forces.structure_forces  FP64 forces -dE/dx by a hand-written reverse pass
  forces.batch_forces      energies and forces of a batch

Every function is pinned by tests in `tests/test_oracle_*.py` against closed
forms, invariances, special cases and independent library routines.  The
absolute energy of a full model is not printed anywhere in the paper (no
worked example, no weights), so whole-model values are pinned only through
those properties.
"""
from .neighbors import CoincidentAtoms, batch_graph, radius_graph  # noqa: F401
from .painn import (batch_energies, cosine_cutoff, gaussian_rbf,  # noqa: F401
                    structure_forward, structure_forward_dense)
