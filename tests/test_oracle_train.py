"""Pins of the training-step oracle (oracle/train.py): the loss gradient
against central differences of the loss built from the already pinned energy
and force oracles, array by array; the complex-step term against a
difference of real weight gradients; invariances of the gradient; heads the
batch does not use; and AdamW against its update written out by hand."""
import numpy as np
import pytest

import synth
from oracle.forces import structure_forces
from oracle.train import COMPLEX_STEP, adamw_step, energy_weight_grad, loss_and_grad


def _model(rbf=0, cap=0, heads=3, seed=11):
    hp = synth.HyperParams(F=6, K=4, L=2, n_species=4, n_heads=heads, cutoff=3.0, shared_dims=[5],
                           branch_dims=[4, 1], rbf_type=rbf, max_neighbors=cap)
    return hp, synth.make_weights(hp, seed)


def _batch(seed=0, heads=(0, 1, 0, 1)):
    rng = np.random.default_rng(seed)
    structs = []
    for k in range(3):
        n = int(rng.integers(3, 6))
        structs.append((rng.uniform(0, 3, (n, 3)), rng.integers(0, 4, n), np.zeros((3, 3)),
                        np.zeros(3, np.uint8), heads[k]))
    Lc = 2.7
    cell = np.array([[Lc, 0, 0], [0.4, Lc, 0], [0.0, -0.3, Lc]])
    structs.append((rng.uniform(0, 1, (3, 3)) @ cell, rng.integers(0, 4, 3), cell, np.ones(3, np.uint8), heads[3]))
    return synth.concat(structs)


def _refs(b, seed=1):
    """Reference energies and forces away from the model's values, so no MAE
    residual is near its kink within the difference step."""
    rng = np.random.default_rng(seed)
    E_ref = rng.standard_normal(b.n_struct) * 3.0 + 5.0
    F_ref = rng.standard_normal((b.n_atoms, 3)) + np.sign(rng.standard_normal((b.n_atoms, 3))) * 4.0
    return E_ref, F_ref


def _loss(b, hp, W, E_ref, F_ref, lam):
    """The loss (R30) from the energy and force oracles alone."""
    E, Fo = [], []
    for k in range(b.n_struct):
        pos, z, cell, pbc, d = b.structure(k)
        o = structure_forces(pos, z, cell, pbc, int(d), hp, W)
        E.append(o["E"])
        Fo.append(o["F"])
    return np.mean(np.abs(np.array(E) - E_ref)) + lam * np.mean(np.abs(np.concatenate(Fo) - F_ref))


@pytest.mark.parametrize("rbf,cap,lam", [(0, 0, 94.8), (1, 3, 94.8), (0, 0, 0.0)])
def test_loss_gradient_matches_central_differences(rbf, cap, lam):
    hp, W = _model(rbf, cap)
    b = _batch()
    E_ref, F_ref = _refs(b)
    o = loss_and_grad(b, hp, W, E_ref, F_ref, lam)
    assert abs(o["loss"] - _loss(b, hp, W, E_ref, F_ref, lam)) <= 1e-12 * o["loss"]
    rng = np.random.default_rng(5)

    def central(k, D, h):
        Wp = dict(W)
        Wm = dict(W)
        Wp[k] = W[k] + h * D
        Wm[k] = W[k] - h * D
        return (_loss(b, hp, Wp, E_ref, F_ref, lam) - _loss(b, hp, Wm, E_ref, F_ref, lam)) / (2 * h)

    h = 2e-5
    for k in W:
        D = rng.standard_normal(W[k].shape)
        # Richardson extrapolation of two central differences: O(h^4)
        fd = (4.0 * central(k, D, h / 2) - central(k, D, h)) / 3.0
        an = float(np.sum(o["grad"][k] * D))
        assert abs(fd - an) <= 1e-8 * max(1.0, abs(fd)), (k, fd, an)


def test_complex_step_equals_difference_of_weight_gradients():
    """Im dE/dtheta(x + i h u) / h against [dE/dtheta(x + eps u) - dE/dtheta(x -
    eps u)] / (2 eps) with real positions, element by element."""
    hp, W = _model()
    b = _batch()
    rng = np.random.default_rng(3)
    pos, z, cell, pbc, d = b.structure(3)
    from oracle.neighbors import radius_graph
    graph = radius_graph(pos, cell, pbc, hp.cutoff)
    u = rng.standard_normal(pos.shape)
    _, Gc = energy_weight_grad(pos + 1j * COMPLEX_STEP * u, z, cell, pbc, int(d), hp, W, graph=graph)
    eps = 1e-6
    _, Gp = energy_weight_grad(pos + eps * u, z, cell, pbc, int(d), hp, W, graph=graph)
    _, Gm = energy_weight_grad(pos - eps * u, z, cell, pbc, int(d), hp, W, graph=graph)
    _, G0 = energy_weight_grad(pos, z, cell, pbc, int(d), hp, W, graph=graph)
    # every array the structure's energy depends on (its own head's branch)
    assert set(W) - set(Gc) == {k for k in W if k.startswith("head") and not k.startswith(f"head{int(d)}.")}
    for k in Gc:
        cs = np.imag(Gc[k]) / COMPLEX_STEP
        fd = (Gp[k] - Gm[k]) / (2 * eps)
        scale = max(1.0, float(np.abs(fd).max()))
        assert np.abs(cs - fd).max() <= 1e-6 * scale, k
        # the real part is the plain weight gradient
        assert np.allclose(np.real(Gc[k]), G0[k], rtol=1e-14, atol=1e-14 * max(1.0, np.abs(G0[k]).max())), k


def test_gradient_invariances():
    """Translating every structure (and moving an atom of the periodic cell
    by a lattice vector) leaves the loss and its gradient unchanged; so does
    reordering the atoms of a structure with its reference forces.  (The
    component-wise force MAE is not invariant under rotation.)"""
    hp, W = _model()
    b = _batch(heads=(0, 1, 2, 0))
    E_ref, F_ref = _refs(b)
    o = loss_and_grad(b, hp, W, E_ref, F_ref, 94.8)
    structs = []
    for k in range(b.n_struct):
        pos, z, cell, pbc, d = b.structure(k)
        pos = pos + np.array([1.0, -2.0, 0.5])
        if np.any(pbc):
            pos = pos.copy()
            pos[1] += cell[0] - cell[2]
        structs.append((pos, z, cell, pbc, d))
    b2 = synth.concat(structs)
    o2 = loss_and_grad(b2, hp, W, E_ref, F_ref, 94.8)
    assert abs(o2["loss"] - o["loss"]) <= 1e-12 * o["loss"]
    for k in W:
        assert np.allclose(o2["grad"][k], o["grad"][k], rtol=0, atol=1e-10 * max(1.0, np.abs(o["grad"][k]).max())), k
    # atom order within structure 0 reversed, with its reference forces
    lo, hi = int(b.struct_ptr[0]), int(b.struct_ptr[1])
    p = np.arange(b.n_atoms)
    p[lo:hi] = p[lo:hi][::-1]
    pos, z, cell, pbc, d = b.structure(0)
    structs = [(pos[::-1], z[::-1], cell, pbc, d)] + [b.structure(k) for k in range(1, b.n_struct)]
    o3 = loss_and_grad(synth.concat(structs), hp, W, E_ref, F_ref[p], 94.8)
    for k in W:
        assert np.allclose(o3["grad"][k], o["grad"][k], rtol=0, atol=1e-11 * max(1.0, np.abs(o["grad"][k]).max())), k


def test_unused_heads_have_zero_gradient():
    hp, W = _model(heads=3)
    b = _batch(heads=(0, 2, 0, 2))
    E_ref, F_ref = _refs(b)
    g = loss_and_grad(b, hp, W, E_ref, F_ref, 94.8)["grad"]
    for k in W:
        if k.startswith("head1."):
            assert np.all(g[k] == 0.0), k
        if k.startswith("head0.") or k.startswith("head2."):
            assert np.any(g[k] != 0.0), k
    # the embedding rows of species absent from the batch get none
    present = set(np.unique(b.species).tolist())
    for sp in range(hp.n_species):
        assert np.any(g["emb"][sp] != 0.0) == (sp in present)


def test_adamw_written_out():
    """Two AdamW steps on two arrays against the update written out with
    scalar arithmetic (decoupled decay, bias-corrected moments)."""
    import math
    W = {"a": np.array([0.5, -2.0]), "b": np.array([[3.0]])}
    G1 = {"a": np.array([0.1, -1e-9]), "b": np.array([[-4.0]])}
    G2 = {"a": np.array([-0.3, 2.0]), "b": np.array([[0.0]])}
    lr, b1, b2, eps, wd = 1e-2, 0.8, 0.95, 1e-6, 0.1
    W1, st = adamw_step(W, G1, {}, lr, b1, b2, eps, wd)
    W2, st = adamw_step(W1, G2, st, lr, b1, b2, eps, wd)
    assert st["t"] == 2

    def by_hand(th, g1, g2):
        m = (1 - b1) * g1
        v = (1 - b2) * g1 * g1
        th = th * (1 - lr * wd) - lr * (m / (1 - b1)) / (math.sqrt(v / (1 - b2)) + eps)
        m = b1 * m + (1 - b1) * g2
        v = b2 * v + (1 - b2) * g2 * g2
        return th * (1 - lr * wd) - lr * (m / (1 - b1 ** 2)) / (math.sqrt(v / (1 - b2 ** 2)) + eps)

    for k in W:
        for idx in np.ndindex(W[k].shape):
            want = by_hand(W[k][idx], G1[k][idx], G2[k][idx])
            assert abs(W2[k][idx] - want) <= 1e-15 * max(1.0, abs(want)), (k, idx)
    # first step: the update is lr * g / (|g| + eps) after the decay
    assert abs(W1["b"][0, 0] - (3.0 * (1 - lr * wd) + lr * 4.0 / (4.0 + eps))) <= 1e-15
