"""Pins of the oracle's PaiNN energy (the lead model's backbone, Table 5)
against closed forms, special cases, symmetries and an independent script.

The paper prints no worked example, so nothing here is a number from it: each
test fixes a property that the mathematics of the method determines."""
import io
import math
import struct

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import synth
from oracle.painn import (cosine_cutoff, gaussian_rbf, structure_forward,
                          structure_forward_dense)

NO_CELL = np.zeros((3, 3))
NO_PBC = np.zeros(3, np.uint8)


def small_hp(F=6, K=7, L=2, S=4, heads=1, shared=(), branch=(3, 1), rc=5.0):
    return synth.HyperParams(F=F, K=K, L=L, n_species=S, n_heads=heads, cutoff=rc,
                             shared_dims=list(shared), branch_dims=list(branch))


def fwd(pos, z, hp, W, cell=NO_CELL, pbc=NO_PBC, ds=0, **kw):
    return structure_forward(np.asarray(pos, float), np.asarray(z), cell, pbc, ds, hp, W, **kw)


# ---------------------------------------------------------------- basis ----
def test_rbf_and_cutoff_closed_forms():
    rc, K = 5.0, 20
    delta = rc / (K - 1)
    mu = np.arange(K) * delta
    g = gaussian_rbf(mu, K, rc)
    assert np.allclose(np.diag(g), 1.0, rtol=0, atol=1e-15)
    # one spacing away from a centre: exp(-1/2); two: exp(-2)
    assert np.isclose(gaussian_rbf(mu[3] + delta, K, rc)[3], math.exp(-0.5), rtol=1e-14)
    assert np.isclose(gaussian_rbf(mu[3] - 2 * delta, K, rc)[3], math.exp(-2.0), rtol=1e-14)
    assert cosine_cutoff(0.0, rc) == 1.0
    assert np.isclose(cosine_cutoff(rc / 2, rc), 0.5, rtol=0, atol=1e-15)
    assert abs(cosine_cutoff(np.nextafter(rc, 0), rc)) < 1e-30
    assert cosine_cutoff(rc, rc) == 0.0 and cosine_cutoff(rc + 1, rc) == 0.0
    # zero slope at r_c: f_c(r_c - h) = (pi h / r_c)^2 / 4 + O(h^4)
    h = 1e-3
    assert np.isclose(cosine_cutoff(rc - h, rc), (math.pi * h / rc) ** 2 / 4, rtol=1e-6)


# ------------------------------------------------- isolated atom, by hand --
def _isolated_energy_from_file(buf: bytes, z: int, head: int) -> float:
    """Independent reading of the weight file for an atom with no neighbours:
    no message, v stays 0, so each layer only adds a^ss([s; 0]) to s."""
    f = io.BytesIO(buf)
    assert f.read(8) == b"PAINNW01"
    F, K, L, S, H, _, ns, nb = struct.unpack("<8i", f.read(32))
    f.read(8)
    shared = struct.unpack(f"<{ns}i", f.read(4 * ns))
    branch = struct.unpack(f"<{nb}i", f.read(4 * nb))
    f.read((-(48 + 4 * ns + 4 * nb)) % 8)
    take = lambda *shape: np.frombuffer(f.read(8 * int(np.prod(shape))), "<f8").reshape(shape)
    act = lambda x: x / (1 + np.exp(-x))
    s = take(S, F)[z]
    for _ in range(L):
        take(F, F), take(F), take(3 * F, F), take(3 * F), take(3 * F, K), take(3 * F)
        take(F, F), take(F, F)
        w1, b1, w2, b2 = take(F, 2 * F), take(F), take(3 * F, F), take(3 * F)
        s = s + (w2 @ act(w1 @ np.concatenate([s, np.zeros(F)]) + b1) + b2)[2 * F:]
    d = F
    for m in range(ns):
        s = act(take(shared[m], d) @ s + take(shared[m])); d = shared[m]
    for h in range(H):
        y = s
        for m in range(nb):
            w, b = take(branch[m], d if m == 0 else branch[m - 1]), take(branch[m])
            y = w @ y + b
            y = act(y) if m < nb - 1 else y
        if h == head:
            out = float(y[0])
    return out


@pytest.mark.parametrize("name", ["tiny_molecules", "screening"])
def test_isolated_atom_matches_independent_script(name):
    hp, W = synth.workload_weights(name)
    buf = synth.weight_file_bytes(hp, W)
    for z, head in [(0, 0), (hp.n_species - 1, hp.n_heads - 1), (3, hp.n_heads // 2)]:
        o = fwd([[1.0, 2.0, 3.0]], [z], hp, W, ds=head)
        want = _isolated_energy_from_file(buf, z, head)
        assert abs(o["E"] - want) <= 1e-12 * abs(want)
        assert np.all(o["v"] == 0)


# ------------------------------------------------------- dimer / cutoff ----
def test_dimer_beyond_cutoff_is_sum_of_isolated_and_continuous():
    hp, W = synth.workload_weights("tiny_molecules")
    rc = hp.cutoff
    e1 = fwd([[0, 0, 0]], [2], hp, W)["E"]
    e2 = fwd([[0, 0, 0]], [7], hp, W)["E"]
    far = fwd([[0, 0, 0], [rc, 0, 0]], [2, 7], hp, W)["E"]
    assert far == pytest.approx(e1 + e2, rel=1e-14)
    gaps = []
    for dlt in [1e-2, 5e-3, 2.5e-3]:
        near = fwd([[0, 0, 0], [rc - dlt, 0, 0]], [2, 7], hp, W)["E"]
        gaps.append(near - (e1 + e2))
    # f_c has zero slope at r_c: the gap is quadratic in delta
    assert gaps[0] / gaps[1] == pytest.approx(4.0, rel=0.02)
    assert gaps[1] / gaps[2] == pytest.approx(4.0, rel=0.02)


# ------------------------------------------------------------ symmetries ----
def _random_molecule(seed, n=9):
    rng = np.random.default_rng(seed)
    b = synth.concat([synth.gen_structure(1234, seed, synth.WORKLOADS["tiny_molecules"])])
    return b.pos, b.species


@pytest.mark.parametrize("seed", range(3))
def test_rotation_reflection_translation_invariance_and_equivariance(seed):
    hp, W = synth.workload_weights("tiny_molecules")
    pos, z = _random_molecule(seed)
    ref = fwd(pos, z, hp, W)
    for k, Q in enumerate([Rotation.random(random_state=seed).as_matrix(),
                           np.diag([1.0, 1.0, -1.0]) @ Rotation.random(random_state=seed + 9).as_matrix()]):
        t = np.array([3.0, -1.5, 0.25]) * (k + 1)
        out = fwd(pos @ Q.T + t, z, hp, W)
        assert out["E"] == pytest.approx(ref["E"], rel=1e-12)
        assert np.allclose(out["s"], ref["s"], rtol=0, atol=1e-11)
        # v_i[c, f] transforms as a polar vector in c (also under reflections)
        assert np.allclose(out["v"], np.einsum("ab,nbf->naf", Q, ref["v"]), rtol=0, atol=1e-11)
    assert np.abs(ref["v"]).max() > 1e-2           # the vector channel is active


@pytest.mark.parametrize("seed", range(2))
def test_permutation_invariance(seed):
    hp, W = synth.workload_weights("tiny_molecules")
    pos, z = _random_molecule(10 + seed)
    ref = fwd(pos, z, hp, W)
    p = np.random.default_rng(seed).permutation(len(z))
    out = fwd(pos[p], z[p], hp, W)
    assert out["E"] == pytest.approx(ref["E"], rel=1e-13)
    assert np.allclose(out["e"], ref["e"][p], rtol=0, atol=1e-12)


def test_linear_and_planar_molecules_keep_vectors_in_their_span():
    hp, W = synth.workload_weights("tiny_molecules")
    line = np.array([[0.0, 0, 0], [1.3, 0, 0], [2.9, 0, 0], [4.1, 0, 0]])
    out = fwd(line, [1, 2, 3, 1], hp, W)
    assert np.abs(out["v"][:, 1:, :]).max() == 0.0 and np.abs(out["v"][:, 0, :]).max() > 1e-3
    plane = np.array([[0.0, 0, 0], [1.3, 0.4, 0], [2.1, -1.2, 0], [0.4, 2.2, 0]])
    out = fwd(plane, [1, 2, 3, 1], hp, W)
    assert np.abs(out["v"][:, 2, :]).max() == 0.0


# ------------------------------------------------------- periodic pins ----
def _periodic(seed, n=6, side=6.5):
    rng = np.random.default_rng(seed)
    while True:
        pos = rng.random((n, 3)) * side
        d = pos[:, None] - pos[None]
        d -= side * np.round(d / side)
        if (np.sqrt((d ** 2).sum(-1)) + np.eye(n) * 9).min() > 1.0:
            return pos, rng.integers(0, 10, n), np.eye(3) * side


def test_lattice_translation_of_an_atom():
    hp, W = synth.workload_weights("tiny_molecules")
    pos, z, cell = _periodic(1)
    pbc = np.ones(3, np.uint8)
    ref = fwd(pos, z, hp, W, cell=cell, pbc=pbc)
    moved = pos.copy()
    moved[2] += 2 * cell[0] - cell[2]
    out = fwd(moved, z, hp, W, cell=cell, pbc=pbc)
    assert out["E"] == pytest.approx(ref["E"], rel=1e-12)


def test_supercell_is_extensive():
    """E(2x2x2 supercell) = 8 E(cell); fails if images beyond the minimum image
    were dropped (the cell is narrower than 2 r_c)."""
    hp, W = synth.workload_weights("tiny_molecules")
    pos, z, cell = _periodic(2, n=5, side=6.0)
    pbc = np.ones(3, np.uint8)
    e1 = fwd(pos, z, hp, W, cell=cell, pbc=pbc)["E"]
    shifts = np.array([[a, b, c] for a in (0, 1) for b in (0, 1) for c in (0, 1)], float)
    big = (pos[None, :, :] + (shifts @ cell)[:, None, :]).reshape(-1, 3)
    e8 = fwd(big, np.tile(z, 8), hp, W, cell=2 * cell, pbc=pbc)["E"]
    assert e8 == pytest.approx(8 * e1, rel=1e-12)


# ------------------------------------------------- two formulations ------
@pytest.mark.parametrize("periodic", [False, True])
def test_loop_form_equals_dense_form(periodic):
    hp, W = synth.workload_weights("tiny_molecules")
    if periodic:
        pos, z, cell = _periodic(3, n=5, side=5.5)
        pbc = np.array([1, 1, 0], np.uint8)
    else:
        pos, z = _random_molecule(21)
        cell, pbc = NO_CELL, NO_PBC
    a = structure_forward(pos, z, cell, pbc, 0, hp, W)
    b = structure_forward_dense(pos, z, cell, pbc, 0, hp, W)
    assert a["E"] == pytest.approx(b["E"], rel=1e-13)
    assert np.allclose(a["v"], b["v"], rtol=0, atol=1e-12)


# ------------------------------------ weight orientation / split pins -----
def _zero_weights(hp):
    return {k: np.zeros(s) for k, s in synth.weight_layout(hp)}


def test_message_split_direction_and_cutoff_on_bias():
    """h = const c (W2phi = 0), filter = f_c(d) * 1 (Wf = 0, bf = 1), identity
    update (a = 0): after one layer a dimer has, in closed form,
    s_1 = Emb + c^s f_c(d) and v_1 = rhat_12 (x) c^r f_c(d) with
    rhat_12 = (x_2 - x_1)/d; after a second layer the sender's vector enters:
    v_1 = rhat_12 (x) c^r f_c (1 - c^v f_c)."""
    F = 3
    hp = small_hp(F=F, K=4, L=2, S=2)
    W = _zero_weights(hp)
    W["emb"] = np.array([[0.1, -0.2, 0.3], [0.5, 0.4, -0.1]])
    c = np.array([1.0, 2.0, 3.0, 0.5, -0.25, 0.125, -1.0, 1.5, 0.75])
    for l in range(2):
        W[f"l{l}.phi_b2"] = c
        W[f"l{l}.filt_b"] = np.ones(3 * F)
    d = 2.2
    x = np.array([[0.3, 0.1, -0.2], [0.3 + d * 0.6, 0.1 + d * 0.8, -0.2]])
    out = fwd(x, [0, 1], hp, W, keep_layers=True)
    fc = 0.5 * (math.cos(math.pi * d / 5.0) + 1)
    rhat = np.array([0.6, 0.8, 0.0])
    s1, v1 = out["layers"][0]
    assert np.allclose(s1[0], W["emb"][0] + c[:F] * fc, atol=1e-14)
    assert np.allclose(v1[0], np.outer(rhat, c[2 * F:] * fc), atol=1e-14)
    assert np.allclose(v1[1], np.outer(-rhat, c[2 * F:] * fc), atol=1e-14)
    s2, v2 = out["layers"][1]
    assert np.allclose(v2[0], np.outer(rhat, c[2 * F:] * fc * (2 - c[F:2 * F] * fc)), atol=1e-14)
    assert np.allclose(s2[0], W["emb"][0] + 2 * c[:F] * fc, atol=1e-14)


def test_filter_orientation_and_rbf_channel():
    """Wf with a single non-zero column k0, bf = 0: the s-message of a dimer is
    c^s * Wf^s[:, k0] * g_k0(d) * f_c(d)."""
    F, K = 2, 5
    hp = small_hp(F=F, K=K, L=1, S=1)
    W = _zero_weights(hp)
    c = np.arange(1, 3 * F + 1, dtype=float)
    W["l0.phi_b2"] = c
    col = np.array([0.5, -1.0, 2.0, 0.25, -0.75, 1.5])
    W["l0.filt_w"][:, 3] = col
    d = 3.1
    out = fwd([[0, 0, 0], [0, 0, d]], [0, 0], hp, W, keep_layers=True)
    g3 = gaussian_rbf(d, K, 5.0)[3]
    fc = cosine_cutoff(d, 5.0)
    assert np.allclose(out["layers"][0][0][0], c[:F] * col[:F] * g3 * fc, atol=1e-15)
    assert np.allclose(out["layers"][0][1][0][2], c[2 * F:] * col[2 * F:] * g3 * fc, atol=1e-15)


def test_phi_orientation():
    """W1phi = permutation P (row f picks input pi(f)), W2phi = [I; 0; 0]:
    h^s_j = silu(s_j[pi(f)]), so a dimer's s-message is silu(s_2[pi(f)]) f_c."""
    F = 4
    hp = small_hp(F=F, K=3, L=1, S=2)
    W = _zero_weights(hp)
    W["emb"] = np.array([[0.2, -0.4, 0.6, 1.1], [-0.3, 0.7, 1.3, -0.9]])
    perm = np.array([2, 0, 3, 1])
    W["l0.phi_w1"][np.arange(F), perm] = 1.0
    W["l0.phi_w2"][:F, :] = np.eye(F)
    W["l0.filt_b"] = np.ones(3 * F)
    d = 1.7
    out = fwd([[0, 0, 0], [d, 0, 0]], [0, 1], hp, W, keep_layers=True)
    silu = lambda x: x / (1 + np.exp(-x))
    fc = cosine_cutoff(d, 5.0)
    assert np.allclose(out["layers"][0][0][0], W["emb"][0] + silu(W["emb"][1][perm]) * fc, atol=1e-15)


def test_update_orientation_and_gate_split():
    """With the message switched off and v set by a first layer, check the
    update block against closed forms for permutation matrices WU / WV and a
    gate that is a constant bias: a = b2a picks [a^vv | a^sv | a^ss]."""
    F = 4
    perm = np.array([1, 2, 3, 0])
    hp = small_hp(F=F, K=3, L=2, S=1)
    base = _zero_weights(hp)
    base["emb"] = np.array([[0.3, -0.1, 0.2, 0.4]])
    # layer 0 creates v = rhat (x) c^r f_c with the identity update
    cr = np.array([1.0, -2.0, 0.5, 3.0])
    base["l0.phi_b2"] = np.concatenate([np.zeros(2 * F), cr])
    base["l0.filt_b"] = np.ones(3 * F)
    d = 2.0
    x = [[0, 0, 0], [0, d, 0]]
    fc = cosine_cutoff(d, 5.0)
    v0 = np.outer([0, 1, 0], cr * fc)                     # atom 0 after layer 0
    s0 = base["emb"][0]

    def run(mod):
        W = {k: v.copy() for k, v in base.items()}
        mod(W)
        return fwd(x, [0, 0], hp, W, keep_layers=True)["layers"][1]

    # a^vv = 1, WU = P: v += P v
    def m1(W):
        W["l1.U"][np.arange(F), perm] = 1.0
        W["l1.upd_b2"][:F] = 1.0
    s, v = run(m1)
    assert np.allclose(v[0], v0 + v0[:, perm], atol=1e-15) and np.allclose(s[0], s0, atol=1e-15)
    # a^sv = 1, WU = P, WV = I: s += sum_c v[c, pi(f)] v[c, f]
    def m2(W):
        W["l1.U"][np.arange(F), perm] = 1.0
        W["l1.V"][:] = np.eye(F)
        W["l1.upd_b2"][F:2 * F] = 1.0
    s, v = run(m2)
    assert np.allclose(s[0], s0 + (v0[:, perm] * v0).sum(0), atol=1e-15)
    # a^ss = silu(n) through W1a = [0 | I], W2a = [0; 0; I], WV = P: n = |v[:, pi(f)]|
    def m3(W):
        W["l1.V"][np.arange(F), perm] = 1.0
        W["l1.upd_w1"][:, F:] = np.eye(F)
        W["l1.upd_w2"][2 * F:, :] = np.eye(F)
    s, v = run(m3)
    silu = lambda t: t / (1 + np.exp(-t))
    assert np.allclose(s[0], s0 + silu(np.abs(v0[1, perm])), atol=1e-15)
    assert np.allclose(v[0], v0, atol=1e-15)


def test_heads_select_dataset_branch():
    hp, W = synth.workload_weights("screening")
    pos = np.array([[0, 0, 0], [1.2, 0, 0], [0, 1.4, 0.3]])
    es = [fwd(pos, [1, 5, 9], hp, W, ds=h)["E"] for h in range(hp.n_heads)]
    assert len(set(np.round(es, 12))) == hp.n_heads
