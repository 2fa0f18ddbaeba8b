"""GPU forward with the lead model's ingredients (Table 5): the Bessel radial
basis and the neighbour cap, vs the FP64 oracle, at all precisions."""
import sys

import numpy as np
import pytest

import synth
from helpers import TOL, check_energies, report_vs_master, stored_weights
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
    Ws = stored_weights(W, precision)
    ref = [structure_forward(*b.structure(k)[:4], 0, hp, Ws) for k in range(b.n_struct)]
    Er = np.array([o["E"] for o in ref])
    Ar = np.array([np.abs(o["e"]).sum() for o in ref])
    check_energies(E, Er, Ar, TOL[precision], f"lead ingredients {precision}")
    if precision == "bf16":
        refm = [structure_forward(*b.structure(k)[:4], 0, hp, W) for k in range(b.n_struct)]
        report_vs_master(E, np.array([o["E"] for o in refm]), np.array([np.abs(o["e"]).sum() for o in refm]), Er,
                         TOL[precision], f"lead ingredients {precision}")
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


@pytest.mark.parametrize("F", [100, 337])
@pytest.mark.parametrize("precision", ["fp64", "fp32", "bf16"])
def test_padded_feature_widths(rt, F, precision):
    """Feature widths the kernels do not run at natively (the lead model's
    F = 337 runs at 384, F = 100 at 128, with zero-padded weights) give the
    energies of the F-wide model."""
    say(f"F = {F}, {precision}")
    hp = synth.HyperParams(F=F, K=4, L=2, n_species=10, n_heads=1, cutoff=5.0,
                           shared_dims=[], branch_dims=[24, 1], rbf_type=RBF_BESSEL)
    W = synth.make_weights(hp, 2200 + F)
    m = rt.load_model(synth.weight_file_bytes(hp, W))
    assert m.info["F"] == F
    b = synth.make_batch("molecules_4096", 0, 24)
    g = rt.build_graph(rt.upload_batch(b), hp.cutoff)
    E = rt.forward(m, g, precision).cpu().numpy()
    ref = [structure_forward(*b.structure(k)[:4], 0, hp, stored_weights(W, precision), keep_layers=True)
           for k in range(b.n_struct)]
    check_energies(E, np.array([o["E"] for o in ref]), np.array([np.abs(o["e"]).sum() for o in ref]),
                   TOL[precision], f"F={F} {precision}")
    if precision == "fp64":
        # the exported features have the model's own width and match layer by layer
        s, v = (t.cpu().numpy() for t in rt.features(m, g, 0, "fp64"))
        assert s.shape == (b.n_atoms, F) and v.shape == (b.n_atoms, 3, F)
        s_ref = np.concatenate([o["layers"][0][0] for o in ref])
        v_ref = np.concatenate([o["layers"][0][1] for o in ref])
        assert np.allclose(s, s_ref, rtol=0, atol=1e-11 * max(1.0, np.abs(s_ref).max()))
        assert np.allclose(v, v_ref, rtol=0, atol=1e-11 * max(1.0, np.abs(v_ref).max()))
    g.free()
    m.free()
