"""The lead-model workload end to end, run exactly as the benchmark runs it:
the lead PaiNN shape (Table "Lead PaiNN model configuration": F = 337, two
layers, four Bessel radial functions, r_c = 5 A, at most 20 neighbours, 16
graph-level branches behind two shared layers of 50 and branch layers of 776,
blended by the branch-weighting MLP), the first 65,536-atom batch of its
stream of 2-500-atom structures (712 structures), one capped graph.  Sampled
structures, always including the largest (494 atoms) and the smallest, are
compared with the FP64 oracle: energies with dataset-id heads and with
blended heads at skip 0.01 in FP64, FP32 and BF16 (BF16 against the oracle
on the BF16-rounded weights, with the error against the master weights
reported beside it); forces with both head modes in FP64 and FP32."""
import sys

import numpy as np
import pytest

import synth
from helpers import (TOL, assert_same_energies, check_blend, check_forces, check_workload_energies, oracle_blend,
                     oracle_forces, report_vs_master)

pytestmark = pytest.mark.gpu

NAME = "lead_model"
SKIP = 0.01
FORCE_TOL = {"fp64": 1e-10, "fp32": 2e-5}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def lead():
    from paper_2604_15380_amd import Runtime
    rt = Runtime(0)
    hp, W = synth.workload_weights(NAME)
    assert (hp.F, hp.L, hp.K, hp.rbf_type, hp.max_neighbors, hp.n_heads) == (337, 2, 4, 1, 20, 16)
    assert hp.shared_dims == [50, 50] and hp.branch_dims == [776, 776, 1] and hp.blend_dims
    m = rt.load_model(synth.weight_file_bytes(hp, W))
    start, cnt = synth.screening_batches(3000, name=NAME)[0]
    b = synth.make_batch(NAME, start, cnt)
    inp = rt.upload_batch(b)
    g = rt.build_graph(inp, hp.cutoff, max_neighbors=hp.max_neighbors)
    n = np.diff(b.struct_ptr)
    rng = np.random.default_rng(61)
    big, small = int(np.argmax(n)), int(np.argmin(n))
    idx_e = sorted(set(rng.choice(b.n_struct, 28, replace=False).tolist()) | {0, b.n_struct - 1, big, small})
    idx_f = sorted(set(rng.choice(b.n_struct, 8, replace=False).tolist()) | {big, small})
    say(f"lead_model batch: {b.n_struct} structures, {b.n_atoms} atoms, {g.n_edges} capped edges; "
        f"largest structure {big} ({n[big]} atoms)")
    yield dict(rt=rt, hp=hp, W=W, m=m, b=b, inp=inp, g=g, idx_e=idx_e, idx_f=idx_f, big=big)
    g.free()
    m.free()
    rt.close()


_cache = {}


def refs(lead, kind):
    """Oracle results, computed once per module: blended energies (on the
    master weights, or on the BF16-rounded weights for "blend_bf16"),
    dataset-id forces, blended forces."""
    if kind not in _cache:
        b = lead["b"]
        say(f"oracle: {kind}")
        if kind == "blend":
            _cache[kind] = oracle_blend(NAME, b, lead["idx_e"], SKIP)
        elif kind == "blend_bf16":
            _cache[kind] = oracle_blend(NAME, b, lead["idx_e"], SKIP, stored="bf16")
        elif kind == "forces":
            _cache[kind] = oracle_forces(NAME, b, lead["idx_f"])
        else:
            _cache[kind] = oracle_forces(NAME, b, lead["idx_f"], blend_skip=SKIP)
    return _cache[kind]


@pytest.mark.parametrize("precision", ["fp64", "fp32", "bf16"])
def test_lead_energies_dataset_heads(lead, precision):
    rt, b, g = lead["rt"], lead["b"], lead["g"]
    say(f"lead_model energies, dataset-id heads, {precision}")
    E = rt.forward(lead["m"], g, precision, dataset_id=lead["inp"]["dataset_id"]).cpu().numpy()
    assert np.all(np.isfinite(E))
    idx = lead["idx_e"]
    check_workload_energies(E[idx], NAME, b, idx, precision, f"lead_model {precision}")


@pytest.mark.parametrize("precision", ["fp64", "fp32", "bf16"])
def test_lead_energies_blended(lead, precision):
    import torch
    rt, b, g, hp = lead["rt"], lead["b"], lead["g"], lead["hp"]
    say(f"lead_model energies, blended heads skip {SKIP}, {precision}")
    w = torch.empty((b.n_struct, hp.n_heads), dtype=torch.float64, device=rt.device)
    E = rt.forward_blend(lead["m"], g, precision, skip=SKIP, weights=w).cpu().numpy()
    w = w.cpu().numpy()
    assert np.all(np.isfinite(E))
    idx = lead["idx_e"]
    ref = refs(lead, "blend_bf16" if precision == "bf16" else "blend")
    check_blend(E, w, ref, idx, SKIP, precision, f"lead_model blended {precision}")
    if precision == "bf16":
        m = refs(lead, "blend")
        report_vs_master(E[idx], np.array([o["E"] for o in m]), np.array([np.abs(o["e"]).sum() for o in m]),
                         np.array([o["E"] for o in ref]), TOL[precision], f"lead_model blended {precision}")


@pytest.mark.parametrize("precision", ["fp64", "fp32"])
def test_lead_forces_dataset_heads(lead, precision):
    rt, b, g = lead["rt"], lead["b"], lead["g"]
    say(f"lead_model forces, dataset-id heads, {precision}")
    E, Fo = rt.forces(lead["m"], g, precision, dataset_id=lead["inp"]["dataset_id"])
    E0 = rt.forward(lead["m"], g, precision, dataset_id=lead["inp"]["dataset_id"])
    assert_same_energies(E.cpu().numpy(), E0.cpu().numpy(), precision)
    Fo = Fo.cpu().numpy()
    check_forces(Fo, b, refs(lead, "forces"), lead["idx_f"], FORCE_TOL[precision], f"lead_model forces {precision}")


@pytest.mark.parametrize("precision", ["fp64", "fp32"])
def test_lead_forces_blended(lead, precision):
    rt, b, g = lead["rt"], lead["b"], lead["g"]
    say(f"lead_model forces, blended heads skip {SKIP}, {precision}")
    E, Fo = rt.forces_blend(lead["m"], g, precision, skip=SKIP)
    E0 = rt.forward_blend(lead["m"], g, precision, skip=SKIP)
    assert_same_energies(E.cpu().numpy(), E0.cpu().numpy(), precision)
    Fo = Fo.cpu().numpy()
    ref = refs(lead, "blend_forces")
    # a head whose weight lies within rounding of the threshold may be kept
    # by one side only: such structures are left out of the comparison
    band = 1e-9 if precision == "fp64" else 1e-5
    ok = [i for i, o in enumerate(ref) if np.all(np.abs(o["w"] - SKIP) > band)]
    idx = [lead["idx_f"][i] for i in ok]
    assert lead["big"] in idx and len(idx) >= len(ref) - 2
    check_forces(Fo, b, [ref[i]["F"] for i in ok], idx, FORCE_TOL[precision],
                 f"lead_model blended forces {precision}")
