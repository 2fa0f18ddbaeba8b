"""Brute-force radius graph (oracle; test infrastructure only).

Defines the neighbour set of the lead model's radius graph (Table 5: cutoff
radius; periodic systems in the fine-tuning section use PBC): every directed
edge (i <- j, n) between atoms i, j of one structure and an integer image
vector n (n_k = 0 on non-periodic axes), except (i, i, 0), whose separation

    t  = (n0*a + n1*b) + n2*c                  (componentwise, cell rows a, b, c)
    r  = (x_j - x_i) + t
    d2 = (r_x*r_x + r_y*r_y) + r_z*r_z

is strictly below r_c*r_c.  Every operation is a separately rounded IEEE
float64 operation in that order, so the set is defined bit-exactly.  All
periodic images within the cutoff are kept (including an atom's own images),
which equals the minimum-image graph whenever each cell width is >= 2 r_c.

Edges are returned sorted by (receiver, sender, n0, n1, n2).  The image range
enumerated here is deliberately generous (a superset of every image that can
hold a neighbour); it does not change the set.

With a neighbour cap (the lead model keeps at most 20 neighbours, Table 5),
each receiver keeps its max_neighbors edges smallest in (d2, sender, n0, n1,
n2) -- the exact d2 above, ties to the lower sender and shift -- and the
kept edges stay in (sender, shift) order (R25).
"""
from __future__ import annotations

import itertools
import math

import numpy as np


class CoincidentAtoms(ValueError):
    """Two distinct atoms (or an atom and a distinct image) at distance 0."""


def cell_widths(cell: np.ndarray) -> np.ndarray:
    """Perpendicular widths |V| / |a_j x a_k| of the cell along each axis."""
    a = np.asarray(cell, dtype=np.float64)
    vol = abs(np.linalg.det(a))
    w = np.empty(3)
    for k in range(3):
        u, v = a[(k + 1) % 3], a[(k + 2) % 3]
        w[k] = vol / np.linalg.norm(np.cross(u, v))
    return w


def image_range(pos: np.ndarray, cell: np.ndarray, pbc, cutoff: float) -> list[int]:
    """Per axis, a bound m_k with every neighbour image inside |n_k| <= m_k.

    For a periodic axis the component of r along the cell normal is
    (f_j - f_i + n_k) * w_k in fractional coordinates f, and it cannot exceed
    |r| < r_c; so |n_k| < r_c / w_k + span_k, with span_k the spread of the
    structure's fractional coordinates.  One extra image is added as margin.
    """
    m = [0, 0, 0]
    if not any(pbc):
        return m
    a = np.asarray(cell, dtype=np.float64)
    frac = np.asarray(pos, dtype=np.float64) @ np.linalg.inv(a)
    w = cell_widths(a)
    for k in range(3):
        if pbc[k]:
            span = float(frac[:, k].max() - frac[:, k].min()) if len(frac) else 0.0
            m[k] = int(math.ceil(cutoff / w[k] + span)) + 1
    return m


def radius_graph(pos, cell, pbc, cutoff: float, max_neighbors: int = 0):
    """All edges of one structure (at most max_neighbors per receiver when > 0).

    Returns (recv, send, shift) with recv/send int64 [E] (structure-local atom
    indices) and shift int64 [E,3], sorted by (recv, send, shift).
    Raises CoincidentAtoms when any candidate pair other than (i, i, 0) is at
    d2 == 0.
    """
    x = np.asarray(pos, dtype=np.float64).reshape(-1, 3)
    n = x.shape[0]
    a = np.asarray(cell, dtype=np.float64).reshape(3, 3)
    rc2 = cutoff * cutoff
    m = image_range(x, a, pbc, cutoff)
    diff = x[None, :, :] - x[:, None, :]          # diff[i, j] = x_j - x_i
    eye = np.eye(n, dtype=bool)
    R, S, T = [], [], []
    for n0, n1, n2 in itertools.product(range(-m[0], m[0] + 1),
                                        range(-m[1], m[1] + 1),
                                        range(-m[2], m[2] + 1)):
        t = (float(n0) * a[0] + float(n1) * a[1]) + float(n2) * a[2]
        r = diff + t
        d2 = (r[..., 0] * r[..., 0] + r[..., 1] * r[..., 1]) + r[..., 2] * r[..., 2]
        keep = d2 < rc2
        if n0 == 0 and n1 == 0 and n2 == 0:
            keep &= ~eye
            zero = (d2 == 0.0) & ~eye
        else:
            zero = d2 == 0.0
        if zero.any():
            i, j = np.argwhere(zero)[0]
            raise CoincidentAtoms(f"atoms {i} and {j} (image {(n0, n1, n2)}) coincide")
        ii, jj = np.nonzero(keep)
        R.append(ii)
        S.append(jj)
        T.append(np.tile(np.array([n0, n1, n2], dtype=np.int64), (len(ii), 1)))
    recv = np.concatenate(R) if R else np.zeros(0, np.int64)
    send = np.concatenate(S) if S else np.zeros(0, np.int64)
    shift = np.concatenate(T) if T else np.zeros((0, 3), np.int64)
    order = np.lexsort((shift[:, 2], shift[:, 1], shift[:, 0], send, recv))
    recv, send, shift = recv[order].astype(np.int64), send[order].astype(np.int64), shift[order]
    if max_neighbors > 0:
        recv, send, shift = cap_neighbors(x, a, recv, send, shift, max_neighbors)
    return recv, send, shift


def cap_neighbors(x, a, recv, send, shift, max_neighbors: int):
    """Keep, per receiver, the max_neighbors edges smallest in (d2, sender,
    shift); the result keeps the input's (receiver, sender, shift) order."""
    r = edge_vectors(x, a, recv, send, shift)
    d2 = (r[:, 0] * r[:, 0] + r[:, 1] * r[:, 1]) + r[:, 2] * r[:, 2]
    order = np.lexsort((shift[:, 2], shift[:, 1], shift[:, 0], send, d2, recv))
    rank = np.empty(len(recv), np.int64)
    first = np.searchsorted(recv[order], recv[order], side="left")
    rank[order] = np.arange(len(recv)) - first
    keep = rank < max_neighbors
    return recv[keep], send[keep], shift[keep]


def edge_vectors(pos, cell, recv, send, shift) -> np.ndarray:
    """r for each edge, by the same expression as the neighbour test."""
    x = np.asarray(pos, dtype=np.float64).reshape(-1, 3)
    a = np.asarray(cell, dtype=np.float64).reshape(3, 3)
    s = shift.astype(np.float64)
    t = (s[:, 0:1] * a[0][None, :] + s[:, 1:2] * a[1][None, :]) + s[:, 2:3] * a[2][None, :]
    return (x[send] - x[recv]) + t


def batch_graph(batch, cutoff: float, max_neighbors: int = 0):
    """Radius graph of a whole batch as a CSR with batch-global atom indices:
    (row_ptr int64 [N+1], col int64 [E], shift int64 [E,3])."""
    N = batch.n_atoms
    cols, shifts, counts = [], [], np.zeros(N, dtype=np.int64)
    for b in range(batch.n_struct):
        lo = int(batch.struct_ptr[b])
        pos, _, cell, pbc, _ = batch.structure(b)
        recv, send, shift = radius_graph(pos, cell, pbc, cutoff, max_neighbors)
        np.add.at(counts, recv + lo, 1)
        cols.append(send + lo)
        shifts.append(shift)
    row_ptr = np.zeros(N + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum(counts)
    col = np.concatenate(cols) if cols else np.zeros(0, np.int64)
    shift = np.concatenate(shifts) if shifts else np.zeros((0, 3), np.int64)
    return row_ptr, col, shift
