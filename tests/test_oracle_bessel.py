"""Pins of the Bessel radial basis (lead model, Table 5) in the oracle:
closed-form values, its orthogonality on [0, r_c] with weight d^2, the
small-distance limit, and the model run with it by both formulations and
under rotation."""
import math

import numpy as np
from scipy.spatial.transform import Rotation

import synth
from oracle.painn import (RBF_BESSEL, bessel_rbf, radial_basis, structure_forward,
                          structure_forward_dense)


def test_closed_form_values():
    rc, K = 5.0, 4
    g = bessel_rbf(np.array([rc / 2]), K, rc)[0]
    assert np.allclose(g, [2 / rc, 0.0, -2 / rc, 0.0], rtol=0, atol=1e-15)
    d = 1.3
    assert np.allclose(bessel_rbf(np.array([d]), K, rc)[0],
                       [math.sin(n * math.pi * d / rc) / d for n in range(1, K + 1)], rtol=1e-15)
    # d -> 0: sin(n pi d / r_c) / d -> n pi / r_c
    assert np.allclose(bessel_rbf(np.array([1e-9]), K, rc)[0], np.arange(1, K + 1) * math.pi / rc, rtol=1e-12)
    assert np.array_equal(radial_basis(np.array([d]), K, rc, RBF_BESSEL), bessel_rbf(np.array([d]), K, rc))


def test_orthogonal_with_weight_d_squared():
    rc, K = 4.0, 6
    x, w = np.polynomial.legendre.leggauss(200)
    d = 0.5 * rc * (x + 1)
    G = bessel_rbf(d, K, rc)
    M = (G * (0.5 * rc * w * d * d)[:, None]).T @ G
    assert np.allclose(M, np.eye(K) * rc / 2, atol=1e-12)


def _bessel_model():
    hp = synth.HyperParams(F=8, K=4, L=2, n_species=5, n_heads=1, cutoff=3.5,
                           shared_dims=[], branch_dims=[4, 1], rbf_type=RBF_BESSEL)
    return hp, synth.make_weights(hp, 91)


def test_bessel_model_two_formulations_and_rotation():
    hp, W = _bessel_model()
    rng = np.random.default_rng(4)
    pos = rng.uniform(0, 3.0, (7, 3))
    z = rng.integers(0, 5, 7)
    cell, pbc = np.zeros((3, 3)), np.zeros(3, np.uint8)
    a = structure_forward(pos, z, cell, pbc, 0, hp, W)
    b = structure_forward_dense(pos, z, cell, pbc, 0, hp, W)
    assert a["n_edges"] > 0
    assert abs(a["E"] - b["E"]) <= 1e-12 * max(1.0, abs(a["E"]))
    Q = Rotation.random(random_state=2).as_matrix()
    c = structure_forward(pos @ Q.T + 1.5, z, cell, pbc, 0, hp, W)
    assert abs(a["E"] - c["E"]) <= 1e-12 * max(1.0, abs(a["E"]))
    # a different basis gives a different energy (the basis is in use)
    hp.rbf_type = 0
    assert abs(structure_forward(pos, z, cell, pbc, 0, hp, W)["E"] - a["E"]) > 1e-6


def test_weight_file_keeps_the_basis_type():
    hp, W = _bessel_model()
    hp2, _ = synth.read_weight_file(synth.weight_file_bytes(hp, W))
    assert hp2.rbf_type == RBF_BESSEL
