"""Pins of the oracle's forces F = -dE/dx (the energy and force pass whose
fused gradient the paper's inference pipeline optimises, Fig. 4).

The reverse pass is checked against quantities it does not compute itself:
central differences of the oracle energy, the closed-form derivatives of the
radial basis and cutoff checked by differences, and the symmetries that fix
forces exactly (no net force, no net torque on a free molecule, rotation
equivariance, action and reaction in a dimer)."""
import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import synth
from oracle.forces import (cosine_cutoff_deriv, radial_basis_deriv, structure_forces)
from oracle.painn import (RBF_BESSEL, RBF_GAUSSIAN, cosine_cutoff, radial_basis,
                          structure_forward)

NO_CELL = np.zeros((3, 3))
NO_PBC = np.zeros(3, np.uint8)


def small_hp(F=6, K=7, L=2, S=4, heads=1, shared=(), branch=(3, 1), rc=5.0, rbf=RBF_GAUSSIAN,
             cap=0):
    return synth.HyperParams(F=F, K=K, L=L, n_species=S, n_heads=heads, cutoff=rc,
                             shared_dims=list(shared), branch_dims=list(branch), rbf_type=rbf,
                             max_neighbors=cap)


def molecule(rng, n, side=3.0):
    while True:
        x = rng.uniform(0, side, (n, 3))
        d = np.linalg.norm(x[:, None] - x[None], axis=-1) + np.eye(n) * 9
        if d.min() > 0.8:
            return x


def energy(x, z, hp, W, cell=NO_CELL, pbc=NO_PBC, ds=0):
    return structure_forward(x, z, cell, pbc, ds, hp, W)["E"]


def central_differences(x, z, hp, W, cell=NO_CELL, pbc=NO_PBC, ds=0, h=1e-5):
    g = np.zeros_like(x)
    for a in range(x.shape[0]):
        for c in range(3):
            xp, xm = x.copy(), x.copy()
            xp[a, c] += h
            xm[a, c] -= h
            g[a, c] = (energy(xp, z, hp, W, cell, pbc, ds) - energy(xm, z, hp, W, cell, pbc, ds)) / (2 * h)
    return -g


@pytest.mark.parametrize("rbf", [RBF_GAUSSIAN, RBF_BESSEL])
def test_basis_and_cutoff_derivatives_by_differences(rbf):
    rc, K, h = 5.0, 9, 1e-6
    d = np.linspace(0.3, 4.9, 37)
    num = (radial_basis(d + h, K, rc, rbf) - radial_basis(d - h, K, rc, rbf)) / (2 * h)
    ana = radial_basis_deriv(d, K, rc, rbf)
    assert np.allclose(ana, num, rtol=1e-7, atol=1e-7 * np.abs(ana).max())
    num = (cosine_cutoff(d + h, rc) - cosine_cutoff(d - h, rc)) / (2 * h)
    assert np.allclose(cosine_cutoff_deriv(d, rc), num, rtol=1e-7, atol=1e-9)
    # zero slope at the cutoff and beyond it
    assert abs(cosine_cutoff_deriv(np.nextafter(rc, 0), rc)) < 1e-15
    assert cosine_cutoff_deriv(rc + 0.1, rc) == 0.0


CASES = {
    "molecule": dict(hp=dict(), periodic=False),
    "molecule_heads": dict(hp=dict(heads=3, shared=(5,), branch=(4, 1), L=3), periodic=False),
    "periodic": dict(hp=dict(rc=3.0), periodic=True),
    "bessel_capped": dict(hp=dict(rbf=RBF_BESSEL, K=4, cap=3), periodic=False),
}


@pytest.mark.parametrize("case", list(CASES))
def test_forces_match_central_differences(case):
    spec = CASES[case]
    hp = small_hp(**spec["hp"])
    W = synth.make_weights(hp, 41)
    rng = np.random.default_rng(7)
    n = 7
    z = rng.integers(0, hp.n_species, n)
    if spec["periodic"]:
        cell = np.diag([3.4, 3.1, 3.7]) + 0.2 * rng.standard_normal((3, 3))
        pbc = np.ones(3, np.uint8)
        x = molecule(rng, n, side=3.0)
    else:
        cell, pbc = NO_CELL, NO_PBC
        x = molecule(rng, n)
    ds = hp.n_heads - 1
    out = structure_forces(x, z, cell, pbc, ds, hp, W)
    assert out["n_edges"] > n
    assert out["E"] == pytest.approx(energy(x, z, hp, W, cell, pbc, ds), rel=1e-13, abs=1e-13)
    num = central_differences(x, z, hp, W, cell, pbc, ds)
    scale = np.abs(out["F"]).max()
    assert scale > 1e-3
    assert np.abs(out["F"] - num).max() <= 2e-7 * scale


def test_no_net_force_or_torque_on_a_molecule():
    hp = small_hp(F=8, L=3)
    W = synth.make_weights(hp, 5)
    rng = np.random.default_rng(11)
    x = molecule(rng, 12, side=4.0)
    z = rng.integers(0, hp.n_species, 12)
    Fo = structure_forces(x, z, NO_CELL, NO_PBC, 0, hp, W)["F"]
    scale = np.abs(Fo).max() * np.abs(x).max()
    assert np.abs(Fo.sum(axis=0)).max() < 1e-12 * np.abs(Fo).max() * 12
    assert np.abs(np.cross(x, Fo).sum(axis=0)).max() < 1e-12 * scale * 12


def test_no_net_force_in_a_periodic_cell():
    hp = small_hp(rc=3.0)
    W = synth.make_weights(hp, 6)
    rng = np.random.default_rng(12)
    x = molecule(rng, 8, side=3.2)
    z = rng.integers(0, hp.n_species, 8)
    cell = np.diag([3.3, 3.3, 3.3])
    Fo = structure_forces(x, z, cell, np.ones(3, np.uint8), 0, hp, W)["F"]
    assert np.abs(Fo.sum(axis=0)).max() < 1e-12 * np.abs(Fo).max() * 8


@pytest.mark.parametrize("seed", [0, 1])
def test_rotation_equivariance(seed):
    hp = small_hp(F=8, L=2)
    W = synth.make_weights(hp, 9)
    rng = np.random.default_rng(seed)
    x = molecule(rng, 9, side=3.5)
    z = rng.integers(0, hp.n_species, 9)
    Q = Rotation.random(random_state=seed).as_matrix()
    F0 = structure_forces(x, z, NO_CELL, NO_PBC, 0, hp, W)["F"]
    F1 = structure_forces(x @ Q.T + 1.5, z, NO_CELL, NO_PBC, 0, hp, W)["F"]
    assert np.abs(F1 - F0 @ Q.T).max() < 1e-12 * np.abs(F0).max() * 10


def test_dimer_action_reaction_along_the_bond():
    hp = small_hp()
    W = synth.make_weights(hp, 3)
    x = np.array([[0.1, 0.2, 0.3], [1.3, 1.9, -0.4]])
    Fo = structure_forces(x, np.array([1, 2]), NO_CELL, NO_PBC, 0, hp, W)["F"]
    u = (x[1] - x[0]) / np.linalg.norm(x[1] - x[0])
    assert np.abs(Fo[0] + Fo[1]).max() < 1e-14 * np.abs(Fo).max() * 4
    assert np.linalg.norm(np.cross(Fo[1], u)) < 1e-13 * np.linalg.norm(Fo[1])
    # an atom beyond the cutoff of both feels nothing
    x3 = np.vstack([x, [[40.0, 0, 0]]])
    F3 = structure_forces(x3, np.array([1, 2, 0]), NO_CELL, NO_PBC, 0, hp, W)["F"]
    assert np.all(F3[2] == 0.0)
    assert np.allclose(F3[:2], Fo, rtol=1e-13, atol=0)


def _blend_hp():
    return synth.HyperParams(F=6, K=5, L=2, n_species=4, n_heads=3, cutoff=5.0, shared_dims=[5],
                             branch_dims=[4, 1], blend_dims=[6])


def test_blended_forces_match_central_differences():
    """Blended heads (section "Composition-conditioned branch weighting"):
    the forces of E = sum_h w_h E_h, with the weights fixed by the
    composition, against differences of the oracle's blended energy."""
    from oracle.forces import structure_forces_blend
    from oracle.painn import structure_forward_blend
    hp = _blend_hp()
    W = synth.make_weights(hp, 77)
    rng = np.random.default_rng(21)
    x = molecule(rng, 7)
    z = rng.integers(0, hp.n_species, 7)
    for skip in (0.0, 0.3):
        out = structure_forces_blend(x, z, NO_CELL, NO_PBC, hp, W, skip=skip)
        E0 = structure_forward_blend(x, z, NO_CELL, NO_PBC, hp, W, skip=skip)["E"]
        assert out["E"] == pytest.approx(E0, rel=1e-13, abs=1e-13)
        h = 1e-5
        num = np.zeros_like(x)
        for a in range(x.shape[0]):
            for c in range(3):
                xp, xm = x.copy(), x.copy()
                xp[a, c] += h
                xm[a, c] -= h
                num[a, c] = -(structure_forward_blend(xp, z, NO_CELL, NO_PBC, hp, W, skip=skip)["E"]
                              - structure_forward_blend(xm, z, NO_CELL, NO_PBC, hp, W, skip=skip)["E"]) / (2 * h)
        assert np.abs(out["F"] - num).max() <= 2e-7 * np.abs(out["F"]).max()


def test_blended_forces_are_the_weighted_head_forces():
    """With the weights of a structure, the blended forces equal the weighted
    sum of the per-head forces (the encoder and the graph are shared)."""
    from oracle.forces import structure_forces_blend
    hp = _blend_hp()
    W = synth.make_weights(hp, 78)
    rng = np.random.default_rng(22)
    x = molecule(rng, 6)
    z = rng.integers(0, hp.n_species, 6)
    out = structure_forces_blend(x, z, NO_CELL, NO_PBC, hp, W)
    per_head = [structure_forces(x, z, NO_CELL, NO_PBC, h, hp, W)["F"] for h in range(hp.n_heads)]
    ref = sum(w * Fh for w, Fh in zip(out["w"], per_head))
    assert np.allclose(out["F"], ref, rtol=1e-12, atol=1e-14)
