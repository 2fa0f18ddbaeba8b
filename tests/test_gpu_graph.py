"""GPU radius graph vs the oracle: the CSR (row_ptr, col, shift) must be
bit-exact, including its order (receiver, sender, shift)."""
import sys

import numpy as np
import pytest

import synth
from oracle.neighbors import batch_graph, radius_graph

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rt():
    from paper_2604_15380_amd import Runtime
    r = Runtime(0)
    yield r
    r.close()


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_csr(rt, batch, cutoff):
    g = rt.build_graph(rt.upload_batch(batch), cutoff)
    try:
        return g.csr()
    finally:
        g.free()


def assert_same_csr(got, want):
    rp, col, sh = got
    wrp, wcol, wsh = want
    assert np.array_equal(rp, wrp)
    assert np.array_equal(col, wcol)
    assert np.array_equal(sh, wsh)


@pytest.mark.parametrize("name", ["tiny_molecules", "molecules_4096"])
def test_molecules_full_batch(rt, name):
    say(f"graph parity {name}")
    b = synth.make_batch(name)
    rc = synth.WORKLOADS[name]["cutoff"]
    assert_same_csr(gpu_csr(rt, b, rc), batch_graph(b, rc))


def test_bulk_full_batch_sampled_rows(rt):
    """All 1024 periodic cells built at once; rows of 40 sampled structures
    compared with the oracle's per-structure graphs."""
    name = "bulk_1024"
    say(f"graph parity {name}")
    b = synth.make_batch(name)
    rc = synth.WORKLOADS[name]["cutoff"]
    rp, col, sh = gpu_csr(rt, b, rc)
    assert rp[-1] == len(col)
    rng = np.random.default_rng(0)
    for s in sorted(set(rng.choice(b.n_struct, 40, replace=False).tolist()) | {0, b.n_struct - 1}):
        lo, hi = int(b.struct_ptr[s]), int(b.struct_ptr[s + 1])
        pos, z, cell, pbc, _ = b.structure(s)
        recv, send, shift = radius_graph(pos, cell, pbc, rc)
        e0, e1 = rp[lo], rp[hi]
        assert e1 - e0 == len(recv), s
        counts = np.bincount(recv, minlength=hi - lo)
        assert np.array_equal(np.diff(rp[lo:hi + 1]), counts)
        assert np.array_equal(col[e0:e1], send + lo)
        assert np.array_equal(sh[e0:e1], shift)
    # ~50-70 neighbours per atom with all images (a stated property of this workload)
    assert 50 <= len(col) / b.n_atoms <= 90


def test_screening_first_batch(rt):
    name = "screening"
    say(f"graph parity {name} first batch")
    start, cnt = synth.screening_batches(3000)[0]
    b = synth.make_batch(name, start, cnt)
    rc = synth.WORKLOADS[name]["cutoff"]
    assert_same_csr(gpu_csr(rt, b, rc), batch_graph(b, rc))


def test_tiny_triclinic_slabs_and_edge_cases(rt):
    say("graph parity: triclinic cells, slabs, empty and single-atom structures")
    rng = np.random.default_rng(5)
    structs = []
    for k in range(24):
        cell = np.eye(3) * (2.4 + rng.random()) + rng.uniform(-0.7, 0.7, (3, 3))
        n = int(rng.integers(1, 6))
        pos = rng.random((n, 3)) @ cell
        if k % 5 == 0:
            pos[0] += 3 * cell[1] - 2 * cell[2]        # outside the home cell
        pbc = np.array([1, 1, k % 2], np.uint8)
        structs.append((pos, rng.integers(0, 4, n), cell, pbc, 0))
    structs.insert(3, (np.zeros((0, 3)), np.zeros(0, np.int32), np.eye(3) * 5, np.ones(3, np.uint8), 0))
    structs.insert(7, (np.array([[0.1, 0.2, 0.3]]), np.array([1]), np.zeros((3, 3)), np.zeros(3, np.uint8), 0))
    structs.append((np.zeros((0, 3)), np.zeros(0, np.int32), np.zeros((3, 3)), np.zeros(3, np.uint8), 0))
    b = synth.concat(structs)
    assert_same_csr(gpu_csr(rt, b, 4.3), batch_graph(b, 4.3))


def test_rebuild_in_place_and_cutoff_boundary(rt):
    say("graph rebuild in place")
    b1 = synth.make_batch("molecules_4096", 0, 300)
    b2 = synth.make_batch("tiny_molecules")
    g = rt.build_graph(rt.upload_batch(b1), 5.0)
    try:
        assert_same_csr(g.csr(), batch_graph(b1, 5.0))
        rt.build_graph(rt.upload_batch(b2), 5.0, graph=g)
        assert_same_csr(g.csr(), batch_graph(b2, 5.0))
        # exactly r_c apart: not an edge; one ulp closer: an edge
        pair = synth.concat([(np.array([[0.0, 0, 0], [5.0, 0, 0]]), np.array([0, 1]), np.zeros((3, 3)),
                              np.zeros(3, np.uint8), 0),
                             (np.array([[0.0, 0, 0], [np.nextafter(5.0, 0), 0, 0]]), np.array([0, 1]),
                              np.zeros((3, 3)), np.zeros(3, np.uint8), 0)])
        rt.build_graph(rt.upload_batch(pair), 5.0, graph=g)
        rp, col, sh = g.csr()
        assert list(rp) == [0, 0, 0, 1, 2] and list(col) == [3, 2]
    finally:
        g.free()


def test_errors(rt):
    from paper_2604_15380_amd import PainnError
    say("graph error paths")
    # coincident atoms
    b = synth.concat([(np.array([[0.0, 0, 0], [1.0, 0, 0], [0.0, 0, 0]]), np.array([0, 1, 2]),
                       np.zeros((3, 3)), np.zeros(3, np.uint8), 0)])
    with pytest.raises(PainnError, match="COINCIDENT"):
        gpu_csr(rt, b, 5.0)
    # an atom on a periodic image of another
    b = synth.concat([(np.array([[0.0, 0, 0], [3.0, 0, 0]]), np.array([0, 1]), np.eye(3) * 3,
                       np.ones(3, np.uint8), 0)])
    with pytest.raises(PainnError, match="COINCIDENT"):
        gpu_csr(rt, b, 2.0)
    # singular periodic cell
    b = synth.concat([(np.array([[0.0, 0, 0], [1.0, 0, 0]]), np.array([0, 1]), np.zeros((3, 3)),
                       np.ones(3, np.uint8), 0)])
    with pytest.raises(PainnError, match="E_ARG"):
        gpu_csr(rt, b, 2.0)
    # malformed struct_ptr
    good = synth.make_batch("tiny_molecules")
    inp = rt.upload_batch(good)
    inp["struct_ptr"][3] = 1000
    with pytest.raises(PainnError, match="E_ARG"):
        rt.build_graph(inp, 5.0)
    # non-positive cutoff
    with pytest.raises(PainnError, match="E_ARG"):
        rt.build_graph(rt.upload_batch(good), 0.0)
    # the context still works after errors
    assert_same_csr(gpu_csr(rt, good, 5.0), batch_graph(good, 5.0))


def _large_structures():
    """Structures large enough for the cell-list search (>= 64 bins of width
    r_c = 5): a molecule, a periodic cube with some atoms stored up to two
    cells outside, a triclinic cell and a flat molecule; plus small molecules
    that keep the all-pairs search in the same batch."""
    rng = np.random.default_rng(5)
    out = []
    n = 900
    a = 2.5 * n ** (1 / 3)
    out.append((rng.uniform(0, a, (n, 3)), np.zeros((3, 3)), np.zeros(3, np.uint8)))
    n = 700
    L = (n / 0.08) ** (1 / 3)
    p = rng.uniform(0, L, (n, 3))
    p[:50] += L * rng.integers(-2, 3, (50, 3))
    out.append((p, np.eye(3) * L, np.ones(3, np.uint8)))
    cell = np.array([[22.0, 0, 0], [4.0, 21.0, 0], [-3.0, 2.5, 23.0]])
    out.append((rng.uniform(0, 1, (600, 3)) @ cell, cell, np.ones(3, np.uint8)))
    p = rng.uniform(0, 40, (500, 3))
    p[:, 2] = 1.0
    out.append((p, np.zeros((3, 3)), np.zeros(3, np.uint8)))
    for _ in range(3):
        n = int(rng.integers(5, 30))
        out.append((rng.uniform(0, 2.5 * n ** (1 / 3), (n, 3)), np.zeros((3, 3)), np.zeros(3, np.uint8)))
    return [(p, rng.integers(0, 10, len(p)).astype(np.int32), c, f, 0) for p, c, f in out]


def test_cell_list_matches_brute_force(rt):
    """The cell-list search gives the oracle's CSR bit for bit (set and order),
    including periodic wraps of atoms stored outside the cell, a triclinic
    cell and a degenerate (flat) bounding box, next to all-pairs structures."""
    say("graph parity: cell lists")
    b = synth.concat(_large_structures())
    assert_same_csr(gpu_csr(rt, b, 5.0), batch_graph(b, 5.0))


def test_cell_list_dense_receivers(rt):
    """Receivers with more neighbours than the fill pass ranks in LDS (a
    dense cluster inside a large sparse molecule) are filled by the all-pairs
    enumeration; the CSR is still the oracle's."""
    say("graph parity: cell list, dense cluster")
    rng = np.random.default_rng(9)
    sparse = rng.uniform(0, 40, (800, 3))
    v = rng.normal(size=(300, 3))
    dense = 20.0 + v / np.linalg.norm(v, axis=1, keepdims=True) * rng.uniform(0, 1, (300, 1)) ** (1 / 3) * 2.4
    pos = np.concatenate([sparse, dense])
    s = (pos, np.zeros(len(pos), np.int32), np.zeros((3, 3)), np.zeros(3, np.uint8), 0)
    b = synth.concat([s])
    rp, col, sh = gpu_csr(rt, b, 5.0)
    assert np.diff(rp).max() > 256
    assert_same_csr((rp, col, sh), batch_graph(b, 5.0))


def gpu_csr_capped(rt, batch, cutoff, cap):
    g = rt.build_graph(rt.upload_batch(batch), cutoff, max_neighbors=cap)
    try:
        return g.csr()
    finally:
        g.free()


@pytest.mark.parametrize("cap", [8, 20])
def test_neighbor_cap_molecules(rt, cap):
    """Lead-model neighbour cap (Table 5: 20): each receiver keeps its nearest
    edges by (d2, sender, shift), in (sender, shift) order, bit for bit."""
    say(f"graph parity: cap {cap}, molecules")
    b = synth.make_batch("molecules_4096", 0, 256)
    assert_same_csr(gpu_csr_capped(rt, b, 5.0, cap), batch_graph(b, 5.0, cap))


def test_neighbor_cap_periodic_and_cell_lists(rt):
    say("graph parity: cap 20, periodic cells; cap 10, cell-list structures")
    b = synth.make_batch("bulk_1024", 0, 12)
    assert_same_csr(gpu_csr_capped(rt, b, 6.0, 20), batch_graph(b, 6.0, 20))
    b = synth.concat(_large_structures())
    assert_same_csr(gpu_csr_capped(rt, b, 5.0, 10), batch_graph(b, 5.0, 10))


def test_neighbor_cap_long_rows(rt):
    """Rows longer than the selection's LDS buffer (a dense cluster)."""
    say("graph parity: cap 20, rows over 256 edges")
    rng = np.random.default_rng(9)
    sparse = rng.uniform(0, 40, (800, 3))
    v = rng.normal(size=(300, 3))
    dense = 20.0 + v / np.linalg.norm(v, axis=1, keepdims=True) * rng.uniform(0, 1, (300, 1)) ** (1 / 3) * 2.4
    pos = np.concatenate([sparse, dense])
    b = synth.concat([(pos, np.zeros(len(pos), np.int32), np.zeros((3, 3)), np.zeros(3, np.uint8), 0)])
    assert_same_csr(gpu_csr_capped(rt, b, 5.0, 20), batch_graph(b, 5.0, 20))
