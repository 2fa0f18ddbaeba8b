"""The C ABI's error paths on a real context: weight files loaded from a path
and the documented failures of painn_model_load (missing file, malformed
contents), null and out-of-range arguments of every entry point, and a graph
whose in-place rebuild failed, which every consumer must refuse on the host
(nothing is launched on it) until a rebuild succeeds."""
import struct
import sys

import numpy as np
import pytest
import torch

import synth
from helpers import TOL

pytestmark = pytest.mark.gpu

E_ARG, E_FILE, E_FORMAT, E_SPECIES, E_COINCIDENT, E_UNSUPPORTED = -1, -4, -5, -6, -7, -8


@pytest.fixture(scope="module")
def rt():
    from paper_2604_15380_amd import Runtime
    r = Runtime(0)
    yield r
    r.close()


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def status_of(fn, *args, **kw):
    from paper_2604_15380_amd import PainnError
    try:
        fn(*args, **kw)
    except PainnError as e:
        return e.status
    return 0


def test_model_load_from_path(rt, tmp_path):
    """painn_model_load reads the same model as painn_model_load_buffer; a
    missing path is PAINN_E_FILE; malformed files are PAINN_E_FORMAT."""
    say("model load from a path")
    hp, W = synth.workload_weights("tiny_molecules")
    data = synth.weight_file_bytes(hp, W)
    p = tmp_path / "tiny.painn"
    p.write_bytes(data)
    m_path = rt.load_model(str(p))
    m_buf = rt.load_model(data)
    assert m_path.info == m_buf.info
    batch = synth.make_batch("tiny_molecules")
    g = rt.build_graph(rt.upload_batch(batch), hp.cutoff)
    E1 = rt.forward(m_path, g, "fp64").cpu().numpy()
    E2 = rt.forward(m_buf, g, "fp64").cpu().numpy()
    assert np.array_equal(E1, E2)
    assert status_of(rt.load_model, str(tmp_path / "missing.painn")) == E_FILE
    for name, bad in [("magic", b"XAINNW01" + data[8:]), ("truncated", data[:-8]),
                      ("trailing", data + b"\0" * 8), ("section", data + b"NBRCAP01" + struct.pack("<2i", 0, 0))]:
        q = tmp_path / f"{name}.painn"
        q.write_bytes(bad)
        assert status_of(rt.load_model, str(q)) == E_FORMAT, name
        assert status_of(rt.load_model, bad) == E_FORMAT, name
    g.free()
    m_path.free()
    m_buf.free()


def test_null_and_bad_arguments(rt):
    """Null array pointers, bad sizes and options are refused with their
    status before anything is launched, and the context keeps working."""
    from paper_2604_15380_amd import binding as B
    say("null and bad arguments")
    hp, W = synth.workload_weights("tiny_molecules")
    model = rt.load_model(synth.weight_file_bytes(hp, W))
    batch = synth.make_batch("tiny_molecules")
    inp = rt.upload_batch(batch)
    g = rt.build_graph(inp, hp.cutoff)
    ctx, mh, gh = rt.ctx, model.handle, g.handle
    sp, pos, spc = inp["struct_ptr"].data_ptr(), inp["pos"].data_ptr(), inp["species"].data_ptr()
    cell, pbc = inp["cell"].data_ptr(), inp["pbc"].data_ptr()
    Bn, Nn = batch.n_struct, batch.n_atoms
    E = torch.empty(Bn, dtype=torch.float64, device=rt.device)
    Fo = torch.empty((Nn, 3), dtype=torch.float64, device=rt.device)
    s = torch.empty((Nn, hp.F), dtype=torch.float64, device=rt.device)
    v = torch.empty((Nn, 3, hp.F), dtype=torch.float64, device=rt.device)
    # graph construction
    bg = lambda *a: B.painn_build_graph(ctx, *a)
    assert status_of(bg, Bn, Nn, None, pos, spc, None, None, hp.cutoff) == E_ARG
    assert status_of(bg, Bn, Nn, sp, None, spc, None, None, hp.cutoff) == E_ARG
    assert status_of(bg, Bn, Nn, sp, pos, None, None, None, hp.cutoff) == E_ARG
    assert status_of(bg, Bn, Nn, sp, pos, spc, None, pbc, hp.cutoff) == E_ARG      # pbc without cell
    assert status_of(bg, -1, Nn, sp, pos, spc, None, None, hp.cutoff) == E_ARG
    assert status_of(bg, 0, Nn, sp, pos, spc, None, None, hp.cutoff) == E_ARG     # atoms, no structures
    assert status_of(bg, Bn, Nn, sp, pos, spc, None, None, float("inf")) == E_ARG
    assert status_of(bg, Bn, Nn, sp, pos, spc, None, None, float("nan")) == E_ARG
    assert status_of(B.painn_build_graph_capped, ctx, Bn, Nn, sp, pos, spc, None, None, hp.cutoff, -1) == E_ARG
    # forward, forces, features
    assert status_of(B.painn_forward, ctx, mh, gh, None, 0, None) == E_ARG
    assert status_of(B.painn_forward, ctx, mh, gh, None, 7, E.data_ptr()) == E_ARG
    assert status_of(B.painn_forward, ctx, None, gh, None, 0, E.data_ptr()) == E_ARG
    assert status_of(B.painn_forward, ctx, mh, None, None, 0, E.data_ptr()) == E_ARG
    assert status_of(B.painn_forces, ctx, mh, gh, None, 0, None, Fo.data_ptr()) == E_ARG
    assert status_of(B.painn_forces, ctx, mh, gh, None, 0, E.data_ptr(), None) == E_ARG
    assert status_of(B.painn_forces, ctx, mh, gh, None, 2, E.data_ptr(), Fo.data_ptr()) == E_UNSUPPORTED
    assert status_of(B.painn_forward_features, ctx, mh, gh, 0, 0, None, v.data_ptr()) == E_ARG
    assert status_of(B.painn_forward_features, ctx, mh, gh, 0, hp.L, s.data_ptr(), v.data_ptr()) == E_ARG
    # the tiny model has no branch-weighting MLP
    assert status_of(B.painn_forward_blend, ctx, mh, gh, 0, 0.0, E.data_ptr(), None) == E_UNSUPPORTED
    # a graph built with another cutoff
    g2 = rt.build_graph(inp, hp.cutoff + 0.5)
    assert status_of(B.painn_forward, ctx, mh, g2.handle, None, 0, E.data_ptr()) == E_ARG
    g2.free()
    # a species index the model does not have
    bad = rt.upload_batch(batch)
    bad["species"][0] = hp.n_species
    g3 = rt.build_graph(bad, hp.cutoff)
    assert status_of(B.painn_forward, ctx, mh, g3.handle, None, 0, E.data_ptr()) == E_SPECIES
    g3.free()
    # profile reads
    assert status_of(B.painn_profile_enable, None, True) == E_ARG
    # the context still works
    from oracle.painn import structure_forward
    Eg = rt.forward(model, g, "fp64").cpu().numpy()
    ref = [structure_forward(*batch.structure(k)[:4], 0, hp, W) for k in range(Bn)]
    Er = np.array([o["E"] for o in ref])
    Ar = np.array([np.abs(o["e"]).sum() for o in ref])
    assert np.max(np.abs(Eg - Er) / Ar) <= TOL["fp64"]
    g.free()
    model.free()


def test_failed_rebuild_leaves_graph_unusable(rt):
    """A graph rebuilt in place from a batch with coincident atoms is refused
    by the forward, the forces and the CSR export (PAINN_E_ARG on the host)
    until a rebuild succeeds; then it gives the right energies again."""
    from paper_2604_15380_amd import binding as B
    say("failed in-place rebuild")
    hp, W = synth.workload_weights("tiny_molecules")
    model = rt.load_model(synth.weight_file_bytes(hp, W))
    good = synth.make_batch("tiny_molecules")
    g = rt.build_graph(rt.upload_batch(good), hp.cutoff)
    E_before = rt.forward(model, g, "fp64").cpu().numpy()
    # the same batch with atom 1 moved onto atom 0: more atoms per structure
    # is not needed, a coincident pair is enough
    pos = good.pos.copy()
    pos[1] = pos[0]
    bad = synth.Batch(pos, good.species, good.struct_ptr, good.cell, good.pbc, good.dataset_id)
    st = status_of(rt.build_graph, rt.upload_batch(bad), hp.cutoff, graph=g)
    assert st == E_COINCIDENT
    E = torch.empty(good.n_struct, dtype=torch.float64, device=rt.device)
    Fo = torch.empty((good.n_atoms, 3), dtype=torch.float64, device=rt.device)
    assert status_of(B.painn_forward, rt.ctx, model.handle, g.handle, None, 0, E.data_ptr()) == E_ARG
    assert status_of(B.painn_forces, rt.ctx, model.handle, g.handle, None, 0, E.data_ptr(),
                     Fo.data_ptr()) == E_ARG
    assert status_of(B.painn_graph_csr, g.handle) == E_ARG
    # a malformed struct_ptr (caught on the device) leaves it unusable too
    inp = rt.upload_batch(good)
    inp["struct_ptr"][3] = 1000
    assert status_of(rt.build_graph, inp, hp.cutoff, graph=g) == E_ARG
    assert status_of(B.painn_forward, rt.ctx, model.handle, g.handle, None, 0, E.data_ptr()) == E_ARG
    # a successful rebuild restores it
    rt.build_graph(rt.upload_batch(good), hp.cutoff, graph=g)
    E_after = rt.forward(model, g, "fp64").cpu().numpy()
    assert np.array_equal(E_before, E_after)
    g.free()
    model.free()
