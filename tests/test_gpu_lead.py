"""GPU forward with the lead model's ingredients (Table 5): the Bessel radial
basis and the neighbour cap, vs the FP64 oracle, at all precisions."""
import sys

import numpy as np
import pytest

import synth
from helpers import TOL, check_energies
from oracle.painn import RBF_BESSEL, structure_forward

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def rt():
    from paper_2604_15380_amd import Runtime
    r = Runtime(0)
    yield r
    r.close()


def _model():
    hp = synth.HyperParams(F=64, K=4, L=3, n_species=10, n_heads=1, cutoff=5.0,
                           shared_dims=[], branch_dims=[32, 1], rbf_type=RBF_BESSEL, max_neighbors=6)
    return hp, synth.make_weights(hp, 2101)


@pytest.mark.parametrize("precision", ["fp64", "fp32", "bf16"])
def test_bessel_capped_model(rt, precision):
    say(f"Bessel basis + neighbour cap, {precision}")
    hp, W = _model()
    m = rt.load_model(synth.weight_file_bytes(hp, W))
    assert m.max_neighbors == 6
    b = synth.make_batch("molecules_4096", 0, 48)
    g = rt.build_graph(rt.upload_batch(b), hp.cutoff, max_neighbors=6)
    E = rt.forward(m, g, precision).cpu().numpy()
    ref = [structure_forward(*b.structure(k)[:4], 0, hp, W) for k in range(b.n_struct)]
    Er = np.array([o["E"] for o in ref])
    Ar = np.array([np.abs(o["e"]).sum() for o in ref])
    check_energies(E, Er, Ar, TOL[precision], f"lead ingredients {precision}")
    g.free()
    m.free()


def test_cap_must_match_the_model(rt):
    from paper_2604_15380_amd import PainnError
    hp, W = _model()
    m = rt.load_model(synth.weight_file_bytes(hp, W))
    b = synth.make_batch("molecules_4096", 0, 4)
    g = rt.build_graph(rt.upload_batch(b), hp.cutoff)          # no cap
    with pytest.raises(PainnError, match="E_ARG"):
        rt.forward(m, g, "fp32")
    g.free()
    m.free()
