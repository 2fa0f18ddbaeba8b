"""GPU forward pass vs the FP64 oracle.

Energies: |E - E_ref| <= tol * sum_i |e_i^ref| per structure with tol =
1e-10 (FP64), 1e-5 (FP32), 2e-2 (BF16).  Small workloads are compared in
full; full-size batches are run whole (as the benchmark runs them) and
compared on sampled structures the oracle evaluates one by one."""
import sys

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import synth
from helpers import TOL, check_energies, check_workload_energies, oracle_energies
from oracle.painn import structure_forward

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


_models = {}


def model(rt, name):
    if name not in _models:
        hp, W = synth.workload_weights(name)
        _models[name] = rt.load_model(synth.weight_file_bytes(hp, W))
    return _models[name]


def run(rt, name, batch, precision, graph=None):
    inp = rt.upload_batch(batch)
    g = rt.build_graph(inp, synth.WORKLOADS[name]["cutoff"])
    ds = inp["dataset_id"] if synth.WORKLOADS[name]["n_heads"] > 1 else None
    E = rt.forward(model(rt, name), g, precision, dataset_id=ds)
    out = E.cpu().numpy()
    g.free()
    return out


@pytest.mark.parametrize("precision", ["fp64", "fp32", "bf16"])
def test_tiny_molecules_all_structures(rt, precision):
    name = "tiny_molecules"
    say(f"forward {name} {precision}")
    b = synth.make_batch(name)
    E = run(rt, name, b, precision)
    norm, rel = check_workload_energies(E, name, b, range(b.n_struct), precision, f"{name} {precision}", workers=1)
    if precision == "fp64":
        assert rel <= 1e-10          # FP64 also meets the plain relative bound


def test_tiny_molecules_features_per_layer(rt):
    """s and v after the embedding and after every layer, FP64, elementwise."""
    name = "tiny_molecules"
    say(f"features {name}")
    b = synth.make_batch(name)
    hp, W = synth.workload_weights(name)
    m = model(rt, name)
    g = rt.build_graph(rt.upload_batch(b), hp.cutoff)
    ref_layers = []
    for k in range(b.n_struct):
        pos, z, cell, pbc, _ = b.structure(k)
        ref_layers.append(structure_forward(pos, z, cell, pbc, 0, hp, W, keep_layers=True)["layers"])
    s0, v0 = rt.features(m, g, -1, "fp64")
    assert np.array_equal(s0.cpu().numpy(), W["emb"][b.species])
    assert not v0.cpu().numpy().any()
    for l in range(hp.L):
        s, v = (t.cpu().numpy() for t in rt.features(m, g, l, "fp64"))
        rs = np.concatenate([ref_layers[k][l][0] for k in range(b.n_struct)])
        rv = np.concatenate([ref_layers[k][l][1] for k in range(b.n_struct)])
        assert np.abs(s - rs).max() <= 1e-11 * np.abs(rs).max(), l
        assert np.abs(v - rv).max() <= 1e-11 * np.abs(rv).max(), l
    g.free()


def _sample(n, k, seed=0):
    rng = np.random.default_rng(seed)
    return sorted(set(rng.choice(n, min(k, n), replace=False).tolist()) | {0, n - 1})


@pytest.mark.parametrize("precision", ["fp32", "bf16", "fp64"])
def test_molecules_4096_full_batch(rt, precision):
    """The benchmark's batch (4096 molecules) in one call; the precision sweep
    runs the same inputs and weights at all three precisions."""
    name = "molecules_4096"
    say(f"forward {name} {precision} (full batch, sampled parity)")
    b = synth.make_batch(name)
    E = run(rt, name, b, precision)
    idx = _sample(b.n_struct, 160)
    check_workload_energies(E[idx], name, b, idx, precision, f"{name} {precision}")


def test_bulk_1024_full_batch_fp64(rt):
    name = "bulk_1024"
    say(f"forward {name} fp64 (full batch, sampled parity)")
    b = synth.make_batch(name)
    E = run(rt, name, b, "fp64")
    idx = _sample(b.n_struct, 22, seed=1)
    Er, Ar = oracle_energies(name, b, idx)
    norm, rel = check_energies(E[idx], Er, Ar, TOL["fp64"], f"{name} fp64")


@pytest.mark.parametrize("precision", ["bf16", "fp32"])
def test_screening_first_batch(rt, precision):
    """One 65,536-atom batch of the screening stream (16 heads by dataset id)."""
    name = "screening"
    say(f"forward {name} {precision} (first batch, sampled parity)")
    start, cnt = synth.screening_batches(3000)[0]
    b = synth.make_batch(name, start, cnt)
    E = run(rt, name, b, precision)
    idx = _sample(b.n_struct, 96, seed=2)
    check_workload_energies(E[idx], name, b, idx, precision, f"{name} {precision}")


def test_screening_stream_sample(rt):
    """The screening stream as the benchmark's stream mode walks it: its
    first 20 batches (about 25,000 structures, each batch closed before
    65,536 atoms), each built and run whole at BF16 and FP32; every 100th
    structure of the stream is compared with the FP64 oracle."""
    name = "screening"
    hp, _ = synth.workload_weights(name)
    m = model(rt, name)
    batches = synth.screening_batches(30000)[:20]
    picked, E_bf16, E_fp32 = [], [], []
    g = None
    for bi, (start, cnt) in enumerate(batches):
        say(f"stream batch {bi}: structures {start}..{start + cnt - 1}")
        b = synth.make_batch(name, start, cnt)
        inp = rt.upload_batch(b)
        g = rt.build_graph(inp, hp.cutoff, graph=g)
        local = [k for k in range(cnt) if (start + k) % 100 == 0]
        for prec, dst in (("bf16", E_bf16), ("fp32", E_fp32)):
            E = rt.forward(m, g, prec, dataset_id=inp["dataset_id"]).cpu().numpy()
            assert np.all(np.isfinite(E)), (bi, prec)
            dst.extend(E[local].tolist())
        picked.extend(b.structure(k) for k in local)
    g.free()
    sample = synth.concat(picked)
    say(f"stream sample: {sample.n_struct} structures of {sum(c for _, c in batches)}")
    check_workload_energies(np.array(E_bf16), name, sample, range(sample.n_struct), "bf16", "screening stream bf16")
    check_workload_energies(np.array(E_fp32), name, sample, range(sample.n_struct), "fp32", "screening stream fp32")


def test_heads_grouping(rt):
    """Atoms are grouped by dataset head before the heads run: one head over
    many tiles, a sparse mix of heads with ragged tile ends, and no dataset ids
    on a 16-head model (head 0 for all) all match the oracle, and a
    structure's energy does not depend on how its batch is grouped."""
    import torch
    name = "screening"
    say("heads grouping")
    start, _ = synth.screening_batches(3000)[0]
    b = synth.make_batch(name, start, 300)
    m = model(rt, name)
    hp, _ = synth.workload_weights(name)
    g = rt.build_graph(rt.upload_batch(b), hp.cutoff)
    rng = np.random.default_rng(11)
    cases = {
        "one head": np.full(b.n_struct, 5, np.int32),
        "sparse mix": rng.choice(np.array([0, 3, 15], np.int32), size=b.n_struct),
    }
    idx = _sample(b.n_struct, 24, seed=4)
    energies = {}
    for label, ds in cases.items():
        bb = synth.Batch(b.pos, b.species, b.struct_ptr, b.cell, b.pbc, ds)
        E = rt.forward(m, g, "fp32", dataset_id=torch.as_tensor(ds, device=rt.device)).cpu().numpy()
        Er, Ar = oracle_energies(name, bb, idx)
        check_energies(E[idx], Er, Ar, TOL["fp32"], f"{name} {label}")
        energies[label] = E
    # no dataset ids: every atom runs head 0
    E0 = rt.forward(m, g, "fp32").cpu().numpy()
    b0 = synth.Batch(b.pos, b.species, b.struct_ptr, b.cell, b.pbc, np.zeros(b.n_struct, np.int32))
    Er, Ar = oracle_energies(name, b0, idx)
    check_energies(E0[idx], Er, Ar, TOL["fp32"], f"{name} no dataset ids")
    # structures on head 5 give the same bits alone in a one-head batch and
    # mixed with other heads
    mix = np.where(cases["sparse mix"] == 15, 5, cases["sparse mix"]).astype(np.int32)
    Em = rt.forward(m, g, "fp32", dataset_id=torch.as_tensor(mix, device=rt.device)).cpu().numpy()
    sel = mix == 5
    assert sel.any()
    assert np.array_equal(Em[sel].view(np.uint64), energies["one head"][sel].view(np.uint64))
    g.free()


def test_invariance_and_equivariance_on_gpu(rt):
    name = "tiny_molecules"
    say("GPU invariance / equivariance")
    b = synth.make_batch(name)
    m = model(rt, name)
    hp, _ = synth.workload_weights(name)
    Q = Rotation.random(random_state=3).as_matrix() @ np.diag([1.0, -1.0, 1.0])
    b2 = synth.Batch(b.pos @ Q.T + np.array([2.0, -7.0, 0.5]), b.species, b.struct_ptr, b.cell, b.pbc,
                     b.dataset_id)
    g1 = rt.build_graph(rt.upload_batch(b), hp.cutoff)
    g2 = rt.build_graph(rt.upload_batch(b2), hp.cutoff)
    E1 = rt.forward(m, g1, "fp64").cpu().numpy()
    E2 = rt.forward(m, g2, "fp64").cpu().numpy()
    assert np.allclose(E1, E2, rtol=1e-12, atol=0)
    s1, v1 = (t.cpu().numpy() for t in rt.features(m, g1, hp.L - 1, "fp64"))
    s2, v2 = (t.cpu().numpy() for t in rt.features(m, g2, hp.L - 1, "fp64"))
    assert np.allclose(s1, s2, rtol=0, atol=1e-11)
    assert np.allclose(v2, np.einsum("ab,nbf->naf", Q, v1), rtol=0, atol=1e-11)
    # permutation of structures within the batch
    p = np.arange(b.n_struct)[::-1]
    g3 = rt.build_graph(rt.upload_batch(b.subset(p)), hp.cutoff)
    E3 = rt.forward(m, g3, "fp64").cpu().numpy()
    assert np.allclose(E3, E1[p], rtol=1e-13, atol=0)
    for g in (g1, g2, g3):
        g.free()


def test_run_to_run_bit_identical(rt):
    name = "molecules_4096"
    say("bitwise reproducibility")
    b = synth.make_batch(name, 0, 512)
    m = model(rt, name)
    g = rt.build_graph(rt.upload_batch(b), 5.0)
    for prec in ("fp32", "bf16", "fp64"):
        a = rt.forward(m, g, prec).cpu().numpy()
        c = rt.forward(m, g, prec).cpu().numpy()
        assert np.array_equal(a.view(np.uint64), c.view(np.uint64)), prec
    g.free()


def test_edge_cases_and_errors(rt):
    from paper_2604_15380_amd import PainnError
    import torch
    say("forward edge cases")
    name = "screening"
    hp, W = synth.workload_weights(name)
    m = model(rt, name)
    from oracle.painn import structure_forward as sf
    structs = [
        (np.zeros((0, 3)), np.zeros(0, np.int32), np.zeros((3, 3)), np.zeros(3, np.uint8), 3),
        (np.array([[0.5, 0.5, 0.5]]), np.array([84]), np.zeros((3, 3)), np.zeros(3, np.uint8), 15),
        (np.array([[0.0, 0, 0], [1.1, 0, 0]]), np.array([7, 7]), np.zeros((3, 3)), np.zeros(3, np.uint8), 0),
        (np.array([[0.3, 0.2, 0.1]]), np.array([5]), np.eye(3) * 2.0, np.ones(3, np.uint8), 9),
    ]
    b = synth.concat(structs)
    inp = rt.upload_batch(b)
    g = rt.build_graph(inp, hp.cutoff)
    E = rt.forward(m, g, "fp32", dataset_id=inp["dataset_id"]).cpu().numpy()
    assert E[0] == 0.0
    for k in (1, 2, 3):
        pos, z, cell, pbc, ds = b.structure(k)
        o = sf(pos, z, cell, pbc, ds, hp, W)
        assert abs(E[k] - o["E"]) <= TOL["fp32"] * np.abs(o["e"]).sum(), k
    # a dataset id outside [0, n_heads) gives NaN for that structure only
    bad = inp["dataset_id"].clone()
    bad[2] = 16
    E = rt.forward(m, g, "fp32", dataset_id=bad).cpu().numpy()
    assert np.isnan(E[2]) and np.isfinite(E[[0, 1, 3]]).all()
    # species outside the model's range
    small = model(rt, "tiny_molecules")      # 10 species
    with pytest.raises(PainnError, match="SPECIES|E_ARG"):
        rt.forward(small, g, "fp32")
    # cutoff mismatch (graph built at 5.0, bulk model uses 6.0)
    with pytest.raises(PainnError, match="E_ARG"):
        rt.forward(model(rt, "bulk_1024"), g, "fp64")
    g.free()
    # an empty batch
    e = synth.concat([])
    ge = rt.build_graph(rt.upload_batch(e), hp.cutoff)
    out = rt.forward(m, ge, "bf16")
    assert out.numel() == 0
    ge.free()


@pytest.mark.parametrize("name", ["bulk_1024", "molecules_4096"])
def test_gaussian_basis_extremes_fp64(rt, name):
    """FP64 forward at the ends of the Gaussian basis the message kernels form
    themselves (K = 32 at 8 k-blocks, K = 20 at 5): edges of 0.05 A (the
    first Gaussians near 1, the last ones near exp(-(K - 1)^2 / 2)), edges
    just inside the cutoff (f_c of order 1e-16 and 1e-8), a chain whose pair
    distances sweep the whole range, and a dense cluster whose receivers
    have more than 16 edges each (chunks shared by several receivers)."""
    hp, W = synth.workload_weights(name)
    rc = hp.cutoff
    z0 = np.zeros((3, 3))
    np0 = np.zeros(3, np.uint8)
    rng = np.random.default_rng(7)
    chain = np.cumsum(np.concatenate([[0.0], [0.05, 0.2, 0.55, 0.9, 1.3, 0.7, 0.35, 1.6, 0.8, 1.1]]))
    cluster = []
    while len(cluster) < 40:      # 20-39 neighbours per atom
        p = rng.uniform(-2.6, 2.6, 3)
        if all(np.linalg.norm(p - q) > 0.9 for q in cluster):
            cluster.append(p)
    structs = [
        (np.array([[0.0, 0, 0], [0.05, 0, 0]]), np.array([3, 5], np.int32), z0, np0, 0),
        (np.array([[0.0, 0, 0], [rc * (1 - 1e-9), 0, 0]]), np.array([2, 2], np.int32), z0, np0, 0),
        (np.array([[0.0, 0, 0], [0, rc - 1e-4, 0]]), np.array([1, 4], np.int32), z0, np0, 0),
        (np.stack([chain, 0.1 * np.sin(chain), np.zeros_like(chain)], 1), (np.arange(len(chain)) % 9 + 1).astype(np.int32),
         z0, np0, 0),
        (np.array(cluster), (np.arange(40) % 7 + 1).astype(np.int32), z0, np0, 0),
    ]
    b = synth.concat(structs)
    say(f"forward {name} fp64, Gaussian basis extremes: {b.n_struct} structures, {b.n_atoms} atoms")
    E = run(rt, name, b, "fp64")
    Er, Ar = oracle_energies(name, b, range(b.n_struct), workers=1)
    check_energies(E, Er, Ar, TOL["fp64"], f"{name} fp64 basis extremes")
