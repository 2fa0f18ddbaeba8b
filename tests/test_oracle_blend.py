"""Pins of the oracle's blended heads (composition -> branch weights -> blend).

The blend is pinned against the single-head readout, which the other oracle
tests pin: a one-hot router reproduces one dataset's energy, an all-zero
router gives the plain mean of the heads (softmax of equal logits), and branch
skipping equals the hand-summed kept heads."""
import copy

import numpy as np
import pytest

import synth
from oracle.painn import blend_weights, composition, structure_forward, structure_forward_blend


def small_blend_model():
    hp = synth.HyperParams(F=16, K=6, L=2, n_species=7, n_heads=5, cutoff=4.0,
                           shared_dims=[8], branch_dims=[12, 1], blend_dims=[10])
    return hp, synth.make_weights(hp, 77)


def structure(seed=3, n=9):
    rng = np.random.default_rng(seed)
    pos = rng.uniform(0, 4.0, (n, 3))
    z = rng.integers(0, 7, n)
    return pos, z, np.zeros((3, 3)), np.zeros(3, np.uint8)


def test_composition_vector():
    z = np.array([3, 1, 3, 3, 0, 6])
    c = composition(z, 7)
    assert c.shape == (7,) and abs(c.sum() - 1.0) < 1e-15
    assert np.array_equal(c * 6, [1, 1, 0, 3, 0, 0, 1])
    assert np.array_equal(composition(z[::-1], 7), c)
    assert np.array_equal(composition(np.zeros(0, int), 7), np.zeros(7))


def test_one_hot_router_is_one_dataset():
    hp, W = small_blend_model()
    pos, z, cell, pbc = structure()
    for k in range(hp.n_heads):
        W2 = copy.deepcopy(W)
        for m in range(len(hp.blend_dims) + 1):
            W2[f"blend{m}.w"][:] = 0.0
            W2[f"blend{m}.b"][:] = 0.0
        W2[f"blend{len(hp.blend_dims)}.b"][k] = 60.0     # exp(-60) * n_heads < 2^-53
        o = structure_forward_blend(pos, z, cell, pbc, hp, W2)
        ref = structure_forward(pos, z, cell, pbc, k, hp, W2)["E"]
        assert o["w"][k] == 1.0
        assert abs(o["E"] - ref) <= 1e-14 * max(1.0, abs(ref))


def test_zero_router_is_the_mean_of_heads():
    hp, W = small_blend_model()
    pos, z, cell, pbc = structure(seed=5)
    for m in range(len(hp.blend_dims) + 1):
        W[f"blend{m}.w"][:] = 0.0
        W[f"blend{m}.b"][:] = 0.0
    o = structure_forward_blend(pos, z, cell, pbc, hp, W)
    assert np.all(o["w"] == 1.0 / hp.n_heads)
    heads = [structure_forward(pos, z, cell, pbc, h, hp, W)["E"] for h in range(hp.n_heads)]
    assert np.allclose(o["E_heads"], heads, rtol=0, atol=1e-13)
    assert abs(o["E"] - np.mean(heads)) <= 1e-13 * max(1.0, np.abs(heads).max())


def test_branch_skipping_keeps_the_heavy_heads():
    hp, W = small_blend_model()
    W[f"blend{len(hp.blend_dims)}.w"] *= 8.0          # a sharper router
    pos, z, cell, pbc = structure(seed=8)
    full = structure_forward_blend(pos, z, cell, pbc, hp, W)
    w = full["w"]
    assert abs(w.sum() - 1.0) < 1e-15
    tau = float(np.sort(w)[hp.n_heads // 2])          # keep the upper half
    o = structure_forward_blend(pos, z, cell, pbc, hp, W, skip=tau)
    heads = [structure_forward(pos, z, cell, pbc, h, hp, W)["E"] for h in range(hp.n_heads)]
    kept = sum(w[h] * heads[h] for h in range(hp.n_heads) if w[h] >= tau)
    assert abs(o["E"] - kept) <= 1e-13 * max(1.0, abs(kept))
    assert abs(full["E"] - sum(w[h] * heads[h] for h in range(hp.n_heads))) <= 1e-13 * max(1.0, abs(kept))
    # nothing kept above the largest weight
    assert structure_forward_blend(pos, z, cell, pbc, hp, W, skip=1.5)["E"] == 0.0


def test_weights_are_permutation_invariant_and_stable():
    hp, W = small_blend_model()
    pos, z, cell, pbc = structure(seed=9)
    p = np.random.default_rng(1).permutation(len(z))
    a = structure_forward_blend(pos, z, cell, pbc, hp, W)
    b = structure_forward_blend(pos[p], z[p], cell, pbc, hp, W)
    assert np.array_equal(a["w"], b["w"])
    assert abs(a["E"] - b["E"]) <= 1e-12 * max(1.0, abs(a["E"]))
    W[f"blend{len(hp.blend_dims)}.b"][:] = 1e3 * np.arange(hp.n_heads)
    w = blend_weights(composition(z, hp.n_species), hp, W)
    assert np.all(np.isfinite(w)) and w[-1] == 1.0


def test_weight_file_round_trip_with_router():
    hp, W = small_blend_model()
    hp2, W2 = synth.read_weight_file(synth.weight_file_bytes(hp, W))
    assert hp2.blend_dims == hp.blend_dims
    assert set(W2) == set(W) and all(np.array_equal(W[k], W2[k]) for k in W)
    hp.blend_dims = None
    Wn = {k: v for k, v in W.items() if not k.startswith("blend")}
    hp3, W3 = synth.read_weight_file(synth.weight_file_bytes(hp, Wn))
    assert hp3.blend_dims is None and not any(k.startswith("blend") for k in W3)


def test_router_hidden_layers_closed_form():
    """The branch-weighting MLP with two hidden layers and hand-chosen
    non-square weights, evaluated by hand with scalar arithmetic: SiLU after
    each hidden layer, none after the output layer, weights applied as
    [out, in], then a softmax.  A dropped or extra SiLU, a transposed layer or
    a missing bias changes the weights far beyond the tolerance."""
    import math
    hp = synth.HyperParams(F=4, K=2, L=1, n_species=3, n_heads=3, cutoff=4.0,
                           shared_dims=[], branch_dims=[1], blend_dims=[4, 2])
    W = synth.make_weights(hp, 5)
    W["blend0.w"] = np.array([[1.0, 0, 0], [0, 2.0, 0], [0, 0, -3.0], [1.0, 1.0, 1.0]])
    W["blend0.b"] = np.array([0.5, -1.0, 0.0, 0.25])
    W["blend1.w"] = np.array([[0.0, 1.0, 0.0, 2.0], [-1.0, 0.0, 1.0, 0.0]])
    W["blend1.b"] = np.array([0.1, -0.2])
    W["blend2.w"] = np.array([[1.0, 0.0], [0.0, 1.0], [2.0, -1.0]])
    W["blend2.b"] = np.array([0.0, 0.3, -0.1])
    z = np.array([0, 0, 1, 2, 2, 2])
    c = composition(z, 3)

    def silu(x):
        return x / (1.0 + math.exp(-x))

    c0, c1, c2 = 2 / 6, 1 / 6, 3 / 6
    h1 = [silu(c0 + 0.5), silu(2 * c1 - 1.0), silu(-3 * c2), silu(c0 + c1 + c2 + 0.25)]
    h2 = [silu(h1[1] + 2 * h1[3] + 0.1), silu(-h1[0] + h1[2] - 0.2)]
    logit = [h2[0], h2[1] + 0.3, 2 * h2[0] - h2[1] - 0.1]
    m = max(logit)
    ex = [math.exp(x - m) for x in logit]
    want = np.array([x / sum(ex) for x in ex])
    got = blend_weights(c, hp, W)
    assert np.allclose(got, want, rtol=1e-14, atol=0), (got, want)
    # the weights are not near-uniform, so the pin has teeth
    assert want.max() - want.min() > 0.2
