"""The synthetic generators: determinism, the stated size / density / distance
recipe, and the weight file round trip."""
import math

import numpy as np
import pytest

import synth


def test_deterministic_and_streams_independent():
    a = synth.make_batch("molecules_4096", 10, 5)
    b = synth.make_batch("molecules_4096", 10, 5)
    assert np.array_equal(a.pos, b.pos) and np.array_equal(a.species, b.species)
    # structure k does not depend on where the batch starts
    c = synth.make_batch("molecules_4096", 12, 1)
    assert np.array_equal(c.pos, a.structure(2)[0])


@pytest.mark.parametrize("name", ["tiny_molecules", "molecules_4096", "bulk_1024", "screening"])
def test_recipe(name):
    spec = synth.WORKLOADS[name]
    b = synth.make_batch(name, 0, 24)
    sizes = np.diff(b.struct_ptr)
    assert sizes.min() >= spec["n_lo"] and sizes.max() <= spec["n_hi"]
    assert b.species.min() >= 0 and b.species.max() < spec["n_species"]
    for s in range(b.n_struct):
        pos, z, cell, pbc, ds = b.structure(s)
        n = len(z)
        d = pos[:, None, :] - pos[None, :, :]
        if pbc.any():
            side = (n / 0.08) ** (1 / 3)
            assert np.allclose(cell, np.eye(3) * side)
            d -= side * np.round(d / side)
            dmin = 1.0
            assert pos.min() >= 0 and pos.max() < side
        else:
            assert not cell.any()
            dmin = 0.9
            assert pos.min() >= 0 and pos.max() < 2.5 * n ** (1 / 3)
        dist = np.sqrt((d ** 2).sum(-1)) + np.eye(n) * 1e9
        assert dist.min() >= dmin
        assert 0 <= ds < spec["n_heads"]


def test_loguniform_sizes_and_batching():
    sizes = synth.stream_sizes("screening", 4000)
    assert sizes.min() >= 4 and sizes.max() <= 200
    # log-uniform: mean of ln n near the mean of U(ln 4, ln 201) minus the floor bias
    assert abs(np.mean(np.log(sizes + 0.5)) - (math.log(4) + math.log(201)) / 2) < 0.1
    batches = synth.screening_batches(4000)
    assert batches[0][0] == 0 and sum(c for _, c in batches) == 4000
    for start, cnt in batches:
        assert sizes[start:start + cnt].sum() <= 65536


def test_weight_file_round_trip(tmp_path):
    hp, w = synth.workload_weights("screening")
    p = tmp_path / "w.bin"
    synth.write_weight_file(str(p), hp, w)
    hp2, w2 = synth.read_weight_file(str(p))
    assert hp2 == hp
    assert list(w2) == list(w)
    assert all(np.array_equal(w[k], w2[k]) for k in w)
    # 11F^2 + 3FK + 11F parameters per layer
    F, K = hp.F, hp.K
    per_layer = sum(w[k].size for k in w if k.startswith("l0."))
    assert per_layer == 11 * F * F + 3 * F * K + 11 * F
    # init scale: N(0, 1/fan_in) (filter: extra gain)
    assert abs(np.std(w["l0.U"]) * math.sqrt(F) - 1) < 0.02
    assert abs(np.std(w["l0.filt_w"]) * math.sqrt(K) / synth.FILTER_GAIN - 1) < 0.05
