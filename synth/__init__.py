"""Seeded synthetic inputs: atomistic batches, model hyperparameters, weights.

This module is the only code shared by the CPU oracle and the GPU library's
tests and benchmark.  It draws random numbers and packs arrays; it holds none
of the model's arithmetic (no neighbour test, no basis function, no layer).

The paper's training and screening corpora (Table 1; the 1.1-billion-structure
screening set of the section on billion-scale inference) and its trained lead
checkpoint are not available, so every workload here is a synthetic stand-in
with the shapes of those corpora: many small molecules and periodic cells,
concatenated into batches, with species drawn from the element counts the
paper quotes (10 for small organic sets, 85 for the full corpus).

Recipe (one independent random stream per structure, so batches of a long
stream can be regenerated in any order):

* stream of structure k: ``numpy.random.Generator(PCG64(SeedSequence([seed, k])))``;
* draws, in this order: atom count n, molecule/periodic coin (mixed streams
  only), dataset id (multi-head workloads only), species (uniform), positions;
* molecule: cube of side ``2.5 * n**(1/3)`` A, positions uniform, each new atom
  rejected while closer than ``d_min`` to an accepted one; no cell;
* periodic: cubic cell of side ``(n / 0.08)**(1/3)`` A (0.08 atoms/A^3),
  positions uniform in the cell, rejection on the minimum-image distance;
* after 10^4 rejections of one atom the structure's positions restart.

Weights: every dense weight and bias ~ N(0, 1/fan_in), the species embedding
~ N(0, 1), drawn in FP64 in the weight file's array order from
``Generator(PCG64(seed))``; the radial filter's weights and bias are then
scaled by FILTER_GAIN.
"""
from __future__ import annotations

import math
import struct
from dataclasses import dataclass, field

import numpy as np

MAGIC = b"PAINNW01"
RBF_GAUSSIAN = 0
# The radial filter's output multiplies a message that is then summed over the
# receiver's neighbours (about 16 cutoff-weighted ones in these workloads), so
# its effective fan-in is ~16 K rather than K: its weights and bias are drawn
# with an extra gain of 1/sqrt(16).  With gain 1 the random 6-layer bulk model
# diverges (the <Uv, Vv> term feeds |v|^2 back into s), overflowing FP64.
FILTER_GAIN = 0.25
# Optional trailing section of the weight file: the branch-weighting MLP that
# maps a structure's composition to softmax weights over the heads.
BLEND_MAGIC = b"BLENDW01"
# Optional section: a cap on the neighbours kept per receiver (Table 5: 20).
NBRCAP_MAGIC = b"NBRCAP01"
# A trained router is sharp (its teacher signal is one-hot per dataset); the
# synthetic one gets a gain on its output layer so that, as reported for the
# trained one, most branches carry negligible weight (~78 % below 0.01 on the
# screening stream, against ~81 % in the paper).
BLEND_GAIN = 24.0


# --------------------------------------------------------------------------
# workloads
# --------------------------------------------------------------------------
WORKLOADS = {
    # 8 molecules of 5-20 atoms, 10 species, r_c = 5 A, F = 64, 3 layers, 20 RBF.
    "tiny_molecules": dict(
        n_struct=8, kind="molecule", n_lo=5, n_hi=20, size_dist="uniform",
        n_species=10, d_min=0.9, cutoff=5.0, F=64, L=3, K=20,
        shared_dims=[], branch_dims=[32, 1], n_heads=1,
        data_seed=1001, weight_seed=2001, precision="fp64"),
    # 4096 molecules of 10-60 atoms, F = 128, 4 layers, 20 RBF.
    "molecules_4096": dict(
        n_struct=4096, kind="molecule", n_lo=10, n_hi=60, size_dist="uniform",
        n_species=10, d_min=0.9, cutoff=5.0, F=128, L=4, K=20,
        shared_dims=[], branch_dims=[64, 1], n_heads=1,
        data_seed=1002, weight_seed=2002, precision="fp32"),
    # 1024 periodic cubic cells of 32-256 atoms at 0.08 A^-3, 85 species,
    # r_c = 6 A, F = 256, 6 layers, 32 RBF.
    "bulk_1024": dict(
        n_struct=1024, kind="periodic", n_lo=32, n_hi=256, size_dist="uniform",
        n_species=85, d_min=1.0, cutoff=6.0, F=256, L=6, K=32,
        shared_dims=[], branch_dims=[128, 1], n_heads=1,
        data_seed=1003, weight_seed=2003, precision="fp64"),
    # 10^6 structures of 4-200 atoms (log-uniform), half molecules and half
    # periodic cells, 85 species, a dataset id in [0,16) per structure picking
    # one of 16 heads (2 shared layers of width 50, branches 776-776-1, the
    # head shape of the lead model in Table 5); r_c = 5 A, F = 256, 4 layers,
    # 32 RBF; greedy batches of at most 65,536 atoms.
    "screening": dict(
        n_struct=1_000_000, kind="mixed", n_lo=4, n_hi=200, size_dist="loguniform",
        n_species=85, d_min=None, cutoff=5.0, F=256, L=4, K=32,
        shared_dims=[50, 50], branch_dims=[776, 776, 1], n_heads=16, blend_dims=[128, 64],
        batch_atoms=65536, data_seed=1005, weight_seed=2005, precision="bf16"),
    # The lead model's shape (Table 5): F = 337, 2 layers, 4 Bessel functions,
    # r_c = 5 A with at most 20 neighbours, 2 shared head layers of 50 and 16
    # branches of 776, 776, blended by the branch-weighting MLP; structures of
    # 2-500 atoms as in the paper's inference benchmark (40,000 structures).
    "lead_model": dict(
        n_struct=40_000, kind="mixed", n_lo=2, n_hi=500, size_dist="loguniform",
        n_species=85, d_min=None, cutoff=5.0, F=337, L=2, K=4, rbf_type=1, max_neighbors=20,
        shared_dims=[50, 50], branch_dims=[776, 776, 1], n_heads=16, blend_dims=[128, 64],
        batch_atoms=65536, data_seed=1006, weight_seed=2006, precision="fp32"),
}
# The precision sweep runs the 4096-molecule inputs and weights at all three
# precisions; it is the same workload entry.
D_MIN_MOLECULE = 0.9
D_MIN_PERIODIC = 1.0


@dataclass
class HyperParams:
    F: int
    K: int
    L: int
    n_species: int
    n_heads: int
    cutoff: float
    shared_dims: list = field(default_factory=list)
    branch_dims: list = field(default_factory=lambda: [1])
    rbf_type: int = RBF_GAUSSIAN
    # hidden widths of the branch-weighting MLP (composition -> head weights);
    # None: the model has none
    blend_dims: list | None = None
    # neighbours kept per receiver, nearest first (0: every neighbour)
    max_neighbors: int = 0

    @staticmethod
    def from_workload(name: str) -> "HyperParams":
        w = WORKLOADS[name]
        bd = w.get("blend_dims")
        return HyperParams(F=w["F"], K=w["K"], L=w["L"], n_species=w["n_species"],
                           n_heads=w["n_heads"], cutoff=w["cutoff"],
                           shared_dims=list(w["shared_dims"]),
                           branch_dims=list(w["branch_dims"]),
                           rbf_type=w.get("rbf_type", RBF_GAUSSIAN),
                           blend_dims=None if bd is None else list(bd),
                           max_neighbors=w.get("max_neighbors", 0))


@dataclass
class Batch:
    """Many structures concatenated.  Shapes: pos [N,3] f64, species [N] i32,
    struct_ptr [B+1] i32, cell [B,3,3] f64 (rows are lattice vectors; zeros for
    molecules), pbc [B,3] u8, dataset_id [B] i32."""
    pos: np.ndarray
    species: np.ndarray
    struct_ptr: np.ndarray
    cell: np.ndarray
    pbc: np.ndarray
    dataset_id: np.ndarray

    @property
    def n_struct(self) -> int:
        return int(self.struct_ptr.shape[0] - 1)

    @property
    def n_atoms(self) -> int:
        return int(self.pos.shape[0])

    def structure(self, b: int):
        lo, hi = int(self.struct_ptr[b]), int(self.struct_ptr[b + 1])
        return (self.pos[lo:hi], self.species[lo:hi], self.cell[b],
                self.pbc[b], int(self.dataset_id[b]))

    def subset(self, idx) -> "Batch":
        """A new batch made of the listed structures, in the listed order."""
        return concat([self.structure(int(b)) for b in idx])


def concat(structs) -> Batch:
    """Pack (pos, species, cell, pbc, dataset_id) tuples into one batch."""
    sizes = [len(s[1]) for s in structs]
    ptr = np.zeros(len(structs) + 1, dtype=np.int32)
    ptr[1:] = np.cumsum(sizes)
    pos = (np.concatenate([np.asarray(s[0], dtype=np.float64).reshape(-1, 3) for s in structs])
           if structs else np.zeros((0, 3)))
    species = (np.concatenate([np.asarray(s[1], dtype=np.int32) for s in structs])
               if structs else np.zeros(0, np.int32))
    cell = np.array([np.asarray(s[2], dtype=np.float64).reshape(3, 3) for s in structs],
                    dtype=np.float64).reshape(-1, 3, 3)
    pbc = np.array([np.asarray(s[3], dtype=np.uint8).reshape(3) for s in structs],
                   dtype=np.uint8).reshape(-1, 3)
    dsid = np.array([int(s[4]) for s in structs], dtype=np.int32)
    return Batch(np.ascontiguousarray(pos), np.ascontiguousarray(species, dtype=np.int32),
                 ptr, np.ascontiguousarray(cell), np.ascontiguousarray(pbc),
                 dsid)


# --------------------------------------------------------------------------
# structure generators
# --------------------------------------------------------------------------
def _stream(seed: int, k: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, k])))


def _positions(rng: np.random.Generator, n: int, side: float, d_min: float,
               periodic: bool) -> np.ndarray:
    d2min = d_min * d_min
    while True:
        pos = np.empty((n, 3), dtype=np.float64)
        m = 0
        ok = True
        while m < n:
            tries = 0
            while True:
                cand = rng.random(3) * side
                if m == 0:
                    break
                d = pos[:m] - cand
                if periodic:
                    d -= side * np.round(d / side)
                if np.min(np.einsum("ij,ij->i", d, d)) >= d2min:
                    break
                tries += 1
                if tries >= 10_000:
                    ok = False
                    break
            if not ok:
                break
            pos[m] = cand
            m += 1
        if ok:
            return pos


def gen_structure(seed: int, k: int, spec: dict):
    """Structure k of a workload's stream: (pos, species, cell, pbc, dataset_id)."""
    rng = _stream(seed, k)
    lo, hi = spec["n_lo"], spec["n_hi"]
    if spec["size_dist"] == "uniform":
        n = int(rng.integers(lo, hi + 1))
    else:  # log-uniform on [lo, hi]: floor(exp(U(ln lo, ln(hi+1))))
        n = int(math.floor(math.exp(rng.uniform(math.log(lo), math.log(hi + 1)))))
        n = min(max(n, lo), hi)
    kind = spec["kind"]
    if kind == "mixed":
        periodic = bool(rng.random() < 0.5)
    else:
        periodic = kind == "periodic"
    dsid = int(rng.integers(0, spec["n_heads"])) if spec["n_heads"] > 1 else 0
    species = rng.integers(0, spec["n_species"], size=n).astype(np.int32)
    if periodic:
        side = (n / 0.08) ** (1.0 / 3.0)
        d_min = spec["d_min"] if spec["d_min"] is not None else D_MIN_PERIODIC
        pos = _positions(rng, n, side, d_min, True)
        cell = np.eye(3) * side
        pbc = np.ones(3, np.uint8)
    else:
        side = 2.5 * n ** (1.0 / 3.0)
        d_min = spec["d_min"] if spec["d_min"] is not None else D_MIN_MOLECULE
        pos = _positions(rng, n, side, d_min, False)
        cell = np.zeros((3, 3))
        pbc = np.zeros(3, np.uint8)
    return pos, species, cell, pbc, dsid


def make_batch(name: str, start: int = 0, count: int | None = None,
               seed: int | None = None) -> Batch:
    """Structures [start, start+count) of a workload's stream as one batch."""
    spec = WORKLOADS[name]
    seed = spec["data_seed"] if seed is None else seed
    if count is None:
        count = spec["n_struct"] - start
    return concat([gen_structure(seed, k, spec) for k in range(start, start + count)])


def stream_sizes(name: str, count: int, seed: int | None = None) -> np.ndarray:
    """Atom counts of the first `count` structures (cheap: only the first draw)."""
    spec = WORKLOADS[name]
    seed = spec["data_seed"] if seed is None else seed
    out = np.empty(count, dtype=np.int64)
    lo, hi = spec["n_lo"], spec["n_hi"]
    for k in range(count):
        rng = _stream(seed, k)
        if spec["size_dist"] == "uniform":
            out[k] = int(rng.integers(lo, hi + 1))
        else:
            n = int(math.floor(math.exp(rng.uniform(math.log(lo), math.log(hi + 1)))))
            out[k] = min(max(n, lo), hi)
    return out


def screening_batches(count: int, name: str = "screening", max_atoms: int | None = None):
    """Greedy batches over the first `count` structures of a stream: a batch is
    closed before it would exceed `max_atoms`.  Returns [(start, n_struct)]."""
    spec = WORKLOADS[name]
    max_atoms = spec.get("batch_atoms", 65536) if max_atoms is None else max_atoms
    sizes = stream_sizes(name, count)
    out, start, atoms = [], 0, 0
    for k, n in enumerate(sizes):
        if atoms + n > max_atoms and k > start:
            out.append((start, k - start))
            start, atoms = k, 0
        atoms += int(n)
    if count > start:
        out.append((start, count - start))
    return out


# --------------------------------------------------------------------------
# weights and the weight file
# --------------------------------------------------------------------------
def weight_layout(hp: HyperParams):
    """(name, shape) of every array of the weight file, in file order.
    Dense weights are stored [out, in] (row = output channel)."""
    F, K = hp.F, hp.K
    out = [("emb", (hp.n_species, F))]
    for l in range(hp.L):
        out += [
            (f"l{l}.phi_w1", (F, F)), (f"l{l}.phi_b1", (F,)),
            (f"l{l}.phi_w2", (3 * F, F)), (f"l{l}.phi_b2", (3 * F,)),
            (f"l{l}.filt_w", (3 * F, K)), (f"l{l}.filt_b", (3 * F,)),
            (f"l{l}.U", (F, F)), (f"l{l}.V", (F, F)),
            (f"l{l}.upd_w1", (F, 2 * F)), (f"l{l}.upd_b1", (F,)),
            (f"l{l}.upd_w2", (3 * F, F)), (f"l{l}.upd_b2", (3 * F,)),
        ]
    d_in = F
    for m, d in enumerate(hp.shared_dims):
        out += [(f"shared{m}.w", (d, d_in)), (f"shared{m}.b", (d,))]
        d_in = d
    for h in range(hp.n_heads):
        di = d_in
        for m, d in enumerate(hp.branch_dims):
            out += [(f"head{h}.{m}.w", (d, di)), (f"head{h}.{m}.b", (d,))]
            di = d
    if hp.blend_dims is not None:
        di = hp.n_species
        for m, d in enumerate(list(hp.blend_dims) + [hp.n_heads]):
            out += [(f"blend{m}.w", (d, di)), (f"blend{m}.b", (d,))]
            di = d
    return out


def make_weights(hp: HyperParams, seed: int) -> dict:
    """FP64 weights keyed by name (insertion order = file order)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w = {}
    layout = weight_layout(hp)
    fan_in = {}
    for name, shape in layout:
        if name.endswith("w1") or name.endswith("w2") or name.endswith(".w") \
                or name.endswith("filt_w") or name.endswith(".U") or name.endswith(".V"):
            fan_in[name] = shape[1]
    for name, shape in layout:
        if name == "emb":
            w[name] = rng.standard_normal(shape)
        elif name in fan_in:
            w[name] = rng.standard_normal(shape) / math.sqrt(fan_in[name])
        else:
            # a bias: same fan-in as the weight just before it in file order
            wname = _bias_partner(name)
            w[name] = rng.standard_normal(shape) / math.sqrt(fan_in[wname])
        if ".filt_" in name:
            w[name] = w[name] * FILTER_GAIN
        if hp.blend_dims is not None and name.startswith(f"blend{len(hp.blend_dims)}."):
            w[name] = w[name] * BLEND_GAIN
    return w


def _bias_partner(bname: str) -> str:
    if bname.endswith("phi_b1"):
        return bname[:-2] + "w1"
    if bname.endswith("phi_b2"):
        return bname[:-2] + "w2"
    if bname.endswith("filt_b"):
        return bname[:-1] + "w"
    if bname.endswith("upd_b1"):
        return bname[:-2] + "w1"
    if bname.endswith("upd_b2"):
        return bname[:-2] + "w2"
    if bname.endswith(".b"):
        return bname[:-1] + "w"
    raise KeyError(bname)


def weight_file_bytes(hp: HyperParams, weights: dict) -> bytes:
    """Serialise: magic 'PAINNW01'; int32 F, K, L, n_species, n_heads, rbf_type,
    n_shared, n_branch; float64 cutoff; int32 shared_dims; int32 branch_dims;
    zero padding to a multiple of 8 bytes; then every array of
    `weight_layout` as little-endian float64, row-major."""
    hdr = MAGIC + struct.pack("<8i", hp.F, hp.K, hp.L, hp.n_species, hp.n_heads,
                              hp.rbf_type, len(hp.shared_dims), len(hp.branch_dims))
    hdr += struct.pack("<d", float(hp.cutoff))
    hdr += struct.pack(f"<{len(hp.shared_dims)}i", *hp.shared_dims)
    hdr += struct.pack(f"<{len(hp.branch_dims)}i", *hp.branch_dims)
    hdr += b"\0" * ((-len(hdr)) % 8)
    parts = [hdr]
    for name, shape in weight_layout(hp):
        if name == "blend0.w":
            # optional section: magic 'BLENDW01'; int32 n_hidden, hidden dims;
            # zero padding to 8 bytes; then the blend arrays
            bh = BLEND_MAGIC + struct.pack("<i", len(hp.blend_dims))
            bh += struct.pack(f"<{len(hp.blend_dims)}i", *hp.blend_dims)
            bh += b"\0" * ((-len(bh)) % 8)
            parts.append(bh)
        a = np.ascontiguousarray(weights[name], dtype="<f8")
        if a.shape != tuple(shape):
            raise ValueError(f"{name}: shape {a.shape} != {shape}")
        parts.append(a.tobytes())
    if hp.max_neighbors > 0:
        # optional section: magic 'NBRCAP01'; int32 max_neighbors, int32 0
        parts.append(NBRCAP_MAGIC + struct.pack("<2i", hp.max_neighbors, 0))
    return b"".join(parts)


def write_weight_file(path: str, hp: HyperParams, weights: dict) -> None:
    with open(path, "wb") as f:
        f.write(weight_file_bytes(hp, weights))


def read_weight_file(path_or_bytes) -> tuple[HyperParams, dict]:
    if isinstance(path_or_bytes, (bytes, bytearray)):
        buf = bytes(path_or_bytes)
    else:
        with open(path_or_bytes, "rb") as f:
            buf = f.read()
    if buf[:8] != MAGIC:
        raise ValueError("bad magic")
    F, K, L, S, H, rbf, ns, nb = struct.unpack_from("<8i", buf, 8)
    (cutoff,) = struct.unpack_from("<d", buf, 40)
    off = 48
    shared = list(struct.unpack_from(f"<{ns}i", buf, off)); off += 4 * ns
    branch = list(struct.unpack_from(f"<{nb}i", buf, off)); off += 4 * nb
    off += (-off) % 8
    hp = HyperParams(F=F, K=K, L=L, n_species=S, n_heads=H, cutoff=cutoff,
                     shared_dims=shared, branch_dims=branch, rbf_type=rbf)
    w = {}

    def take(layout):
        nonlocal off
        for name, shape in layout:
            cnt = int(np.prod(shape))
            w[name] = np.frombuffer(buf, dtype="<f8", count=cnt, offset=off).reshape(shape).copy()
            off += 8 * cnt

    take(weight_layout(hp))
    while off < len(buf):
        magic = buf[off:off + 8]
        if magic == BLEND_MAGIC and hp.blend_dims is None:
            (nh,) = struct.unpack_from("<i", buf, off + 8)
            hp.blend_dims = list(struct.unpack_from(f"<{nh}i", buf, off + 12))
            off += 12 + 4 * nh
            off += (-off) % 8
            take([(n, sh) for n, sh in weight_layout(hp) if n.startswith("blend")])
        elif magic == NBRCAP_MAGIC and hp.max_neighbors == 0:
            hp.max_neighbors = struct.unpack_from("<i", buf, off + 8)[0]
            off += 16
        else:
            raise ValueError("trailing bytes in weight file")
    if off != len(buf):
        raise ValueError("trailing bytes in weight file")
    return hp, w


def workload_weights(name: str) -> tuple[HyperParams, dict]:
    hp = HyperParams.from_workload(name)
    return hp, make_weights(hp, WORKLOADS[name]["weight_seed"])
