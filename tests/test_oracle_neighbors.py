"""Pins of the oracle's radius graph against closed forms, scipy's KD-tree and
an independent brute-force image loop (the cutoff radius and PBC handling of
the lead model, Table 5; periodic systems of the fine-tuning section)."""
import itertools

import numpy as np
import pytest
from scipy.spatial import cKDTree

import synth
from oracle.neighbors import CoincidentAtoms, batch_graph, radius_graph


def _edge_set(recv, send, shift):
    return {(int(i), int(j), int(a), int(b), int(c)) for i, j, (a, b, c) in zip(recv, send, shift)}


@pytest.mark.parametrize("seed", range(6))
def test_molecule_pairs_equal_kdtree(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(5, 60))
    pos = rng.random((n, 3)) * 2.5 * n ** (1 / 3)
    rc = 5.0
    recv, send, shift = radius_graph(pos, np.zeros((3, 3)), [0, 0, 0], rc)
    assert np.all(shift == 0)
    pairs = cKDTree(pos).query_pairs(rc)
    want = {(i, j) for i, j in pairs} | {(j, i) for i, j in pairs}
    assert {(int(i), int(j)) for i, j in zip(recv, send)} == want


@pytest.mark.parametrize("seed", range(4))
def test_orthorhombic_min_image_equals_kdtree_boxsize(seed):
    # every cell width > 2 r_c, so the all-images graph is the minimum-image one
    rng = np.random.default_rng(100 + seed)
    L = np.array([11.0, 12.5, 10.5]) + rng.random(3)
    n = 40
    pos = rng.random((n, 3)) * L
    rc = 5.0
    recv, send, shift = radius_graph(pos, np.diag(L), [1, 1, 1], rc)
    pairs = cKDTree(pos, boxsize=L).query_pairs(rc)
    want = {(i, j) for i, j in pairs} | {(j, i) for i, j in pairs}
    got = [(int(i), int(j)) for i, j in zip(recv, send)]
    assert len(got) == len(set(got))          # one image per pair
    assert set(got) == want
    # the image vector reproduces the minimum-image displacement
    r = pos[send] - pos[recv] + shift * L
    mic = pos[send] - pos[recv]
    mic -= L * np.round(mic / L)
    assert np.allclose(r, mic, atol=1e-12)


def _independent_images(pos, cell, pbc, rc, M=4):
    """Plain loops over a fixed image range +-M on periodic axes."""
    out = set()
    n = len(pos)
    rng_ = [range(-M, M + 1) if p else range(0, 1) for p in pbc]
    for i in range(n):
        for j in range(n):
            for a, b, c in itertools.product(*rng_):
                if i == j and a == b == c == 0:
                    continue
                t = (a * cell[0] + b * cell[1]) + c * cell[2]
                r = (pos[j] - pos[i]) + t
                if (r[0] * r[0] + r[1] * r[1]) + r[2] * r[2] < rc * rc:
                    out.add((i, j, a, b, c))
    return out


@pytest.mark.parametrize("seed", range(5))
def test_small_triclinic_cells_equal_independent_loop(seed):
    rng = np.random.default_rng(200 + seed)
    cell = np.eye(3) * (2.6 + rng.random()) + rng.uniform(-0.6, 0.6, (3, 3))
    n = int(rng.integers(1, 5))
    frac = rng.random((n, 3))
    pos = frac @ cell
    pbc = [1, 1, int(seed % 2)]            # also a slab (non-periodic z)
    rc = 4.2
    got = _edge_set(*radius_graph(pos, cell, pbc, rc))
    assert got == _independent_images(pos, cell, pbc, rc, M=5)
    # self images exist for such small cells
    assert any(i == j for i, j, *_ in got)


def test_simple_cubic_shell_counts():
    # one atom in a cubic cell of side a: neighbours are lattice vectors, so the
    # counts are the simple-cubic shells 6, 12, 8 at a, a*sqrt2, a*sqrt3
    a = 2.0
    pos = np.array([[0.3, 0.2, 0.1]])
    cell = np.eye(3) * a
    for rc, want in [(2.5, 6), (3.0, 18), (3.6, 26), (4.1, 32)]:
        recv, send, shift = radius_graph(pos, cell, [1, 1, 1], rc)
        assert len(recv) == want
        d = np.linalg.norm(shift * a, axis=1)
        assert np.all(d < rc)


def test_sorted_by_receiver_sender_shift_and_unwrapped_positions():
    rng = np.random.default_rng(7)
    cell = np.eye(3) * 4.0
    pos = rng.random((6, 3)) * 4.0
    pos[2] += np.array([8.0, -4.0, 12.0])       # far outside the home cell
    recv, send, shift = radius_graph(pos, cell, [1, 1, 1], 4.5)
    key = np.stack([recv, send, shift[:, 0], shift[:, 1], shift[:, 2]], 1)
    assert all(tuple(key[k]) < tuple(key[k + 1]) for k in range(len(key) - 1))
    # moving atom 2 by lattice vectors only relabels its images: same distances
    pos2 = pos.copy()
    pos2[2] -= np.array([8.0, -4.0, 12.0])
    r1 = radius_graph(pos, cell, [1, 1, 1], 4.5)
    r2 = radius_graph(pos2, cell, [1, 1, 1], 4.5)
    assert len(r1[0]) == len(r2[0])


def test_coincident_atoms_raise():
    pos = np.array([[0.0, 0.0, 0.0], [1.0, 0.0, 0.0], [0.0, 0.0, 0.0]])
    with pytest.raises(CoincidentAtoms):
        radius_graph(pos, np.zeros((3, 3)), [0, 0, 0], 5.0)
    # an atom on another's periodic image
    pos = np.array([[0.0, 0.0, 0.0], [3.0, 0.0, 0.0]])
    with pytest.raises(CoincidentAtoms):
        radius_graph(pos, np.eye(3) * 3.0, [1, 1, 1], 2.0)


def test_batch_graph_offsets_and_cutoff_edge_cases():
    b = synth.make_batch("tiny_molecules")
    row_ptr, col, shift = batch_graph(b, 5.0)
    assert row_ptr[0] == 0 and row_ptr[-1] == len(col)
    for s in range(b.n_struct):
        lo, hi = b.struct_ptr[s], b.struct_ptr[s + 1]
        c = col[row_ptr[lo]:row_ptr[hi]]
        assert np.all((c >= lo) & (c < hi))
    # a pair at exactly r_c is not an edge (strict inequality)
    pos = np.array([[0.0, 0.0, 0.0], [5.0, 0.0, 0.0]])
    assert len(radius_graph(pos, np.zeros((3, 3)), [0, 0, 0], 5.0)[0]) == 0
    pos = np.array([[0.0, 0.0, 0.0], [np.nextafter(5.0, 0.0), 0.0, 0.0]])
    assert len(radius_graph(pos, np.zeros((3, 3)), [0, 0, 0], 5.0)[0]) == 2
    # single atom, no pbc: no edges
    assert len(radius_graph(np.zeros((1, 3)), np.zeros((3, 3)), [0, 0, 0], 5.0)[0]) == 0


# ---- neighbour cap (lead model: 20 neighbours, Table 5) ---------------------

def _capped_by_loops(pos, cell, pbc, rc, cap):
    """Independent brute force: every (i, j, n) in a small image box, the
    exact d2, sorted tuples; the `cap` smallest (d2, j, n) per receiver,
    returned in (i, j, n) order."""
    x = np.asarray(pos, float)
    a = np.asarray(cell, float)
    m = [2 if p else 0 for p in pbc]
    edges = []
    for i in range(len(x)):
        cand = []
        for j in range(len(x)):
            for n0 in range(-m[0], m[0] + 1):
                for n1 in range(-m[1], m[1] + 1):
                    for n2 in range(-m[2], m[2] + 1):
                        if i == j and (n0, n1, n2) == (0, 0, 0):
                            continue
                        t = (float(n0) * a[0] + float(n1) * a[1]) + float(n2) * a[2]
                        r = (x[j] - x[i]) + t
                        d2 = (r[0] * r[0] + r[1] * r[1]) + r[2] * r[2]
                        if d2 < rc * rc:
                            cand.append((d2, j, n0, n1, n2))
        for d2, j, n0, n1, n2 in sorted(cand)[:cap]:
            edges.append((i, j, n0, n1, n2))
    edges.sort()
    e = np.array(edges, dtype=np.int64).reshape(-1, 5)
    return e[:, 0], e[:, 1], e[:, 2:]


def test_cap_matches_loops_molecule_and_cell():
    rng = np.random.default_rng(12)
    pos = rng.uniform(0, 5.0, (14, 3))
    for cap in (1, 3, 6):
        got = radius_graph(pos, np.zeros((3, 3)), [0, 0, 0], 3.5, cap)
        want = _capped_by_loops(pos, np.zeros((3, 3)), [0, 0, 0], 3.5, cap)
        for g, w in zip(got, want):
            assert np.array_equal(g, w), cap
    cell = np.array([[4.1, 0, 0], [0.6, 3.9, 0], [0.3, -0.4, 4.4]])
    pos = rng.uniform(0, 1, (6, 3)) @ cell
    got = radius_graph(pos, cell, [1, 1, 1], 3.0, 5)
    want = _capped_by_loops(pos, cell, [1, 1, 1], 3.0, 5)
    for g, w in zip(got, want):
        assert np.array_equal(g, w)


def test_cap_above_degree_changes_nothing_and_ties_go_to_lower_index():
    rng = np.random.default_rng(13)
    pos = rng.uniform(0, 6.0, (30, 3))
    full = radius_graph(pos, np.zeros((3, 3)), [0, 0, 0], 3.0)
    big = radius_graph(pos, np.zeros((3, 3)), [0, 0, 0], 3.0, 1000)
    assert all(np.array_equal(a, b) for a, b in zip(full, big))
    # simple cubic lattice, spacing 1: the centre's 6 nearest are equidistant
    g = np.array([(i, j, k) for i in range(3) for j in range(3) for k in range(3)], float)
    centre = 13
    recv, send, shift = radius_graph(g, np.zeros((3, 3)), [0, 0, 0], 1.2, 3)
    kept = send[recv == centre]
    six = sorted(j for j in range(27) if abs(np.abs(g[j] - g[centre]).sum() - 1.0) < 1e-12)
    assert kept.tolist() == six[:3]
    # periodic: an atom alone in a cubic cell of side 1 has 6 images at distance 1;
    # with cap 2 the lowest shifts in (n0, n1, n2) order are kept
    r, s, t = radius_graph(np.zeros((1, 3)), np.eye(3), [1, 1, 1], 1.2, 2)
    assert t.tolist() == [[-1, 0, 0], [0, -1, 0]]
