"""GPU blended heads (branch-weighting MLP + branch skipping) vs the oracle.

Energies use the tolerance metric of the other forward tests (BF16 against
the oracle on the BF16-rounded weights).  Where the skip threshold decides
whether a head is kept, the two sides compute the weight in different
precisions: a head whose oracle weight lies within the weight tolerance of
the threshold may be kept by one side and not the other, so its
contribution w_h |E_h| is added to that structure's allowed error; every
other head must be kept or skipped alike."""
import copy
import sys

import numpy as np
import pytest

import synth
from helpers import TOL, check_blend, report_vs_master, stored_weights
from oracle.painn import structure_forward, structure_forward_blend

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


@pytest.fixture(scope="module")
def screening(rt):
    name = "screening"
    hp, W = synth.workload_weights(name)
    m = rt.load_model(synth.weight_file_bytes(hp, W))
    start, cnt = synth.screening_batches(3000)[0]
    b = synth.make_batch(name, start, cnt)
    g = rt.build_graph(rt.upload_batch(b), hp.cutoff)
    yield hp, W, m, b, g
    g.free()
    m.free()


def _sample(n, k, seed):
    rng = np.random.default_rng(seed)
    return sorted(set(rng.choice(n, min(k, n), replace=False).tolist()) | {0, n - 1})


@pytest.mark.parametrize("precision,skip", [("bf16", 0.0), ("bf16", 0.01), ("fp32", 0.0), ("fp32", 0.01),
                                            ("fp64", 0.0)])
def test_blend_screening_batch(rt, screening, precision, skip):
    import torch
    hp, W, m, b, g = screening
    say(f"blend {precision} skip={skip}")
    assert m.has_blend
    w_gpu = torch.empty((b.n_struct, hp.n_heads), dtype=torch.float64, device=rt.device)
    E = rt.forward_blend(m, g, precision, skip=skip, weights=w_gpu).cpu().numpy()
    w_gpu = w_gpu.cpu().numpy()
    assert np.all(np.isfinite(E)) and np.allclose(w_gpu.sum(1), 1.0, atol=1e-5 if precision != "bf16" else 1e-3)
    idx = _sample(b.n_struct, 24 if precision == "fp64" else 48, seed=21)
    Ws = stored_weights(W, precision)
    refs = [structure_forward_blend(*b.structure(k)[:4], hp, Ws, skip=skip) for k in idx]
    check_blend(E, w_gpu, refs, idx, skip, precision, f"screening blended {precision} skip {skip}")
    if precision == "bf16":
        master = [structure_forward_blend(*b.structure(k)[:4], hp, W, skip=skip) for k in idx]
        report_vs_master(E[idx], np.array([o["E"] for o in master]), np.array([np.abs(o["e"]).sum() for o in master]),
                         np.array([o["E"] for o in refs]), TOL[precision], f"screening blended {precision}")
    if skip > 0:
        # most heads carry negligible weight (the premise of branch skipping)
        assert (w_gpu < skip).mean() > 0.5


def test_one_hot_router_equals_the_dataset_head(rt):
    """A router that puts all weight on head k gives the energies of the
    single-head forward with every dataset id = k."""
    import torch
    name = "screening"
    hp, W = synth.workload_weights(name)
    start, cnt = synth.screening_batches(3000)[0]
    b = synth.make_batch(name, start, 200)
    g = rt.build_graph(rt.upload_batch(b), hp.cutoff)
    for k in (0, 11):
        W2 = copy.deepcopy(W)
        last = len(hp.blend_dims)
        for mm in range(last + 1):
            W2[f"blend{mm}.w"][:] = 0.0
            W2[f"blend{mm}.b"][:] = 0.0
        W2[f"blend{last}.b"][k] = 60.0
        m = rt.load_model(synth.weight_file_bytes(hp, W2))
        Eb = rt.forward_blend(m, g, "fp32", skip=0.5).cpu().numpy()
        ds = torch.full((b.n_struct,), k, dtype=torch.int32, device=rt.device)
        Ed = rt.forward(m, g, "fp32", dataset_id=ds).cpu().numpy()
        assert np.array_equal(Eb, Ed), k
        m.free()
    g.free()


def test_blend_errors_and_limits(rt, screening):
    from paper_2604_15380_amd import PainnError
    hp, W, m, b, g = screening
    say("blend errors")
    with pytest.raises(PainnError, match="E_ARG"):
        rt.forward_blend(m, g, "fp32", skip=-1.0)
    # every head below the threshold: nothing is kept
    E = rt.forward_blend(m, g, "fp32", skip=1.5).cpu().numpy()
    assert np.all(E == 0.0)
    # a model without a branch-weighting MLP
    hp1, W1 = synth.workload_weights("molecules_4096")
    m1 = rt.load_model(synth.weight_file_bytes(hp1, W1))
    assert not m1.has_blend
    bm = synth.make_batch("molecules_4096", 0, 4)
    gm = rt.build_graph(rt.upload_batch(bm), hp1.cutoff)
    with pytest.raises(PainnError, match="UNSUPPORTED"):
        rt.forward_blend(m1, gm, "fp32")
    gm.free()
    m1.free()
    # an empty batch
    e = synth.concat([])
    ge = rt.build_graph(rt.upload_batch(e), hp.cutoff)
    assert rt.forward_blend(m, ge, "bf16", skip=0.01).numel() == 0
    ge.free()
