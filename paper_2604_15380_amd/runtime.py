"""Torch-facing convenience layer over the C ABI: device memory and the HIP
stream come from torch; every computation runs in libpainn.so."""
from __future__ import annotations

import ctypes

import numpy as np

from . import binding as B


def _hip():
    return ctypes.CDLL("libamdhip64.so")


def copy_from_device(dst, src_ptr: int, nbytes: int) -> None:
    """Copy `nbytes` from a library-owned device pointer into a torch tensor."""
    import torch
    if nbytes == 0:
        return
    torch.cuda.synchronize(dst.device)
    h = _hip()
    h.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    err = h.hipMemcpy(dst.data_ptr(), src_ptr, nbytes, 3)   # hipMemcpyDeviceToDevice
    if err != 0:
        raise RuntimeError(f"hipMemcpy failed ({err})")


class Model:
    def __init__(self, rt: "Runtime", handle: int):
        self.rt, self.handle = rt, handle
        self.info = B.painn_model_info(handle)
        opts = B.painn_model_options(handle)
        self.has_blend = opts["has_blend"]
        self.max_neighbors = opts["max_neighbors"]

    def free(self):
        if self.handle:
            B.painn_model_free(self.handle)
            self.handle = 0


class Graph:
    def __init__(self, rt: "Runtime", handle: int, inputs):
        self.rt, self.handle, self.inputs = rt, handle, inputs
        self.refresh()

    def refresh(self):
        c = B.painn_graph_csr(self.handle)
        self.n_edges, self.n_atoms, self.n_struct = c["n_edges"], c["n_atoms"], c["n_struct"]
        self._ptrs = c

    def csr(self):
        """(row_ptr [N+1], col [E], shift [E,3]) as CPU numpy int64 arrays."""
        import torch
        dev = self.rt.device
        rp = torch.empty(self.n_atoms + 1, dtype=torch.int32, device=dev)
        col = torch.empty(self.n_edges, dtype=torch.int32, device=dev)
        sh = torch.empty(self.n_edges, dtype=torch.int32, device=dev)
        copy_from_device(rp, self._ptrs["row_ptr"], 4 * (self.n_atoms + 1))
        copy_from_device(col, self._ptrs["col"], 4 * self.n_edges)
        copy_from_device(sh, self._ptrs["shift"], 4 * self.n_edges)
        sh_np = sh.cpu().numpy().view(np.int8).reshape(-1, 4)[:, :3].astype(np.int64)
        return rp.cpu().numpy().astype(np.int64), col.cpu().numpy().astype(np.int64), sh_np

    def free(self):
        if self.handle:
            B.painn_graph_free(self.handle)
            self.handle = 0


class Runtime:
    """One library context on a torch CUDA (HIP) device and its current stream."""

    def __init__(self, device: int = 0):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU: the HIP library has no CPU path")
        self.device = torch.device("cuda", device)
        self.stream = torch.cuda.current_stream(self.device)
        self.ctx = B.painn_create(device, self.stream.cuda_stream)

    # ---- inputs ----------------------------------------------------------
    def upload_batch(self, batch):
        """Copy a synth.Batch (numpy) to device tensors."""
        import torch
        d = self.device
        return dict(
            n_struct=batch.n_struct, n_atoms=batch.n_atoms,
            struct_ptr=torch.from_numpy(np.ascontiguousarray(batch.struct_ptr, dtype=np.int32)).to(d),
            pos=torch.from_numpy(np.ascontiguousarray(batch.pos, dtype=np.float64)).to(d),
            species=torch.from_numpy(np.ascontiguousarray(batch.species, dtype=np.int32)).to(d),
            cell=torch.from_numpy(np.ascontiguousarray(batch.cell, dtype=np.float64)).to(d),
            pbc=torch.from_numpy(np.ascontiguousarray(batch.pbc, dtype=np.uint8)).to(d),
            dataset_id=torch.from_numpy(np.ascontiguousarray(batch.dataset_id, dtype=np.int32)).to(d),
            any_pbc=bool(np.any(batch.pbc)),
        )

    # ---- model / graph / forward ----------------------------------------
    def load_model(self, src) -> Model:
        if isinstance(src, (bytes, bytearray)):
            return Model(self, B.painn_model_load_buffer(self.ctx, bytes(src)))
        return Model(self, B.painn_model_load(self.ctx, str(src)))

    def build_graph(self, inp: dict, cutoff: float, graph: Graph | None = None,
                    max_neighbors: int = 0) -> Graph:
        """Radius graph of an uploaded batch; max_neighbors > 0 keeps that
        many nearest neighbours per receiver (a capped model needs its cap)."""
        ptr = lambda t: t.data_ptr() if t is not None and t.numel() else None
        use_pbc = inp.get("any_pbc", True)
        h = B.painn_build_graph_capped(self.ctx, inp["n_struct"], inp["n_atoms"], ptr(inp["struct_ptr"]),
                                       ptr(inp["pos"]), ptr(inp["species"]),
                                       ptr(inp["cell"]) if use_pbc else None,
                                       ptr(inp["pbc"]) if use_pbc else None, cutoff, max_neighbors,
                                       graph.handle if graph else None)
        if graph is not None:
            graph.inputs = inp
            graph.refresh()
            return graph
        return Graph(self, h, inp)

    def forward(self, model: Model, graph: Graph, precision="fp32", dataset_id=None, out=None):
        import torch
        prec = B.PRECISIONS[precision] if isinstance(precision, str) else precision
        if out is None:
            out = torch.empty(graph.n_struct, dtype=torch.float64, device=self.device)
        ds = dataset_id.data_ptr() if dataset_id is not None and dataset_id.numel() else None
        B.painn_forward(self.ctx, model.handle, graph.handle, ds, prec,
                        out.data_ptr() if out.numel() else None)
        return out

    def forward_blend(self, model: Model, graph: Graph, precision="fp32", skip=0.0, out=None,
                      weights=None):
        """Energies with every head blended by the model's branch-weighting
        MLP; heads with weight < skip are left out.  `weights` (optional)
        receives the [B, n_heads] head weights."""
        import torch
        prec = B.PRECISIONS[precision] if isinstance(precision, str) else precision
        if out is None:
            out = torch.empty(graph.n_struct, dtype=torch.float64, device=self.device)
        B.painn_forward_blend(self.ctx, model.handle, graph.handle, prec, skip,
                              out.data_ptr() if out.numel() else None,
                              weights.data_ptr() if weights is not None and weights.numel() else None)
        return out

    def forces(self, model: Model, graph: Graph, precision="fp32", dataset_id=None, energies=None,
               forces=None):
        """Energies [B] and forces -dE/dx [N, 3] (float64) by the reverse pass."""
        import torch
        prec = B.PRECISIONS[precision] if isinstance(precision, str) else precision
        if energies is None:
            energies = torch.empty(graph.n_struct, dtype=torch.float64, device=self.device)
        if forces is None:
            forces = torch.empty((graph.n_atoms, 3), dtype=torch.float64, device=self.device)
        ds = dataset_id.data_ptr() if dataset_id is not None and dataset_id.numel() else None
        B.painn_forces(self.ctx, model.handle, graph.handle, ds, prec,
                       energies.data_ptr() if energies.numel() else None,
                       forces.data_ptr() if forces.numel() else None)
        return energies, forces

    def forces_blend(self, model: Model, graph: Graph, precision="fp32", skip=0.0, energies=None,
                     forces=None, weights=None):
        """Energies and forces with every head blended by the model's
        branch-weighting MLP (heads with weight < skip left out)."""
        import torch
        prec = B.PRECISIONS[precision] if isinstance(precision, str) else precision
        if energies is None:
            energies = torch.empty(graph.n_struct, dtype=torch.float64, device=self.device)
        if forces is None:
            forces = torch.empty((graph.n_atoms, 3), dtype=torch.float64, device=self.device)
        B.painn_forces_blend(self.ctx, model.handle, graph.handle, prec, skip,
                             energies.data_ptr() if energies.numel() else None,
                             forces.data_ptr() if forces.numel() else None,
                             weights.data_ptr() if weights is not None and weights.numel() else None)
        return energies, forces

    def features(self, model: Model, graph: Graph, layer: int, precision="fp64"):
        import torch
        prec = B.PRECISIONS[precision] if isinstance(precision, str) else precision
        F = model.info["F"]
        s = torch.empty((graph.n_atoms, F), dtype=torch.float64, device=self.device)
        v = torch.empty((graph.n_atoms, 3, F), dtype=torch.float64, device=self.device)
        B.painn_forward_features(self.ctx, model.handle, graph.handle, prec, layer,
                                 s.data_ptr() if s.numel() else None,
                                 v.data_ptr() if v.numel() else None)
        return s, v

    def synchronize(self):
        B.painn_synchronize(self.ctx)

    def close(self):
        if self.ctx:
            B.painn_destroy(self.ctx)
            self.ctx = 0
