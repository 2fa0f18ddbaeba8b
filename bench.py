"""Benchmark of the batched PaiNN screening forward pass on one MI355X.

A step is one pass of the whole hot path over one batch already resident in
HBM: radius graph (painn_build_graph) + forward (embedding, L interaction
layers, heads, per-structure energies).  Default workload: 4096 molecules of
10-60 atoms, F = 128, 4 layers, 20 Gaussian RBF, FP32.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "PaiNN forward structures/s and edge-messages/s on 1 MI355X (FP64/FP32/BF16)"
METRIC_FORCES = "PaiNN energy+forces structures/s on 1 MI355X (FP64/FP32)"
# MI355X published peaks (dense), TFLOP/s
PEAK = {
    "alu": {"fp64": 78.6, "fp32": 157.3, "bf16": 157.3},     # vector ALU (BF16 mode computes in FP32)
    "mfma": {"fp64": 78.6, "fp32": 157.3, "bf16": 2500.0},
}
HBM_PEAK_GBS = 8000.0
DTYPE = {"fp64": "f64", "fp32": "f32", "bf16": "bf16"}
ELEM = {"fp64": 8, "fp32": 4, "bf16": 2}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# the kernel sources a stored traffic measurement depends on (per mode)
KERNEL_SOURCES = ["paper_2604_15380_amd/csrc/forward.hip", "paper_2604_15380_amd/csrc/mfma.h",
                  "paper_2604_15380_amd/csrc/neighbors.hip"]
KERNEL_SOURCES_FORCES = KERNEL_SOURCES + ["paper_2604_15380_amd/csrc/backward.hip"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_digest(forces: bool = False) -> str:
    h = hashlib.sha256()
    for p in (KERNEL_SOURCES_FORCES if forces else KERNEL_SOURCES):
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def kernel_work(kernel: str, hp, N: int, E: int, prec: str, head_entries: int | None = None):
    """Algorithmic work of ONE launch of a kernel class: (bound, flops, bytes).

    message: per edge 6KF (radial filter contraction over K Gaussians for 3F
             channels) + 22F (cutoff and bias, scalar and vector messages);
             minimum HBM bytes: per atom h (3F), v in (3F), s (F) read and s
             (F), v out (3F) written, plus 8 bytes of CSR per edge.  The first
             layer's v is zero, so its launch forms 2 of the 3 filter parts
             (4KF), does half the elementwise work (11F) and reads no v; the
             figure per launch is the mean over the L launches.
    update:  per atom 22 F^2 (U/V 12F^2, gate MLP 10F^2) + 8 F^2 for the next
             layer's phi fused behind it (all but the last layer).
    phi:     per atom 8 F^2.
    heads:   per (atom, head) entry the shared and branch MLP flops (one entry
             per atom, or every kept head of the atom's structure when blended).
    Reverse pass (forces):
    bwd_message: per edge 12KF (the filter and its d-derivative) + 36F
             (elementwise terms and the per-edge sums over channels); minimum
             HBM bytes: per atom h, v (6F) and g_s', g_v' (4F) read, g_h, g_v
             (6F) written, plus 8 bytes of CSR per edge.
    bwd_update: per atom 22 F^2 (the transposed products W2a^T, W1a^T and
             [U^T|V^T] for 3 components; U, V, the gate come from the forward).
    bwd_phi: per atom 10 F^2 (W1 s recomputed, W2^T, W1^T).
    bwd_heads: per (atom, head) entry twice the heads' forward flops of every
             layer but the 1-wide output (the pre-activations recomputed, then
             the transposed layers).
    """
    F, K, L = hp.F, hp.K, hp.L
    b = ELEM[prec]
    if kernel == "message":
        fl = E * ((L - 1) * (6.0 * K * F + 22.0 * F) + (4.0 * K * F + 11.0 * F)) / L
        nb = N * ((L - 1) * 11.0 + 8.0) / L * F * b + 8.0 * E
        return "alu", fl, nb
    if kernel == "update":
        fl = N * (22.0 * F * F + 8.0 * F * F * (L - 1) / L)
        return "mfma", fl, N * (8.0 * F + 3.0 * F * (L - 1) / L) * b
    if kernel == "phi":
        return "mfma", N * 8.0 * F * F, N * 4.0 * F * b
    if kernel == "bwd_message":
        ab = 8 if prec == "fp64" else 4
        return "alu", E * (12.0 * K * F + 36.0 * F), N * (6.0 * F * b + 10.0 * F * ab) + 8.0 * E
    if kernel == "bwd_update":
        ab = 8 if prec == "fp64" else 4
        return "mfma", N * 22.0 * F * F, N * (9.0 * F * b + 8.0 * F * ab)
    if kernel == "bwd_phi":
        ab = 8 if prec == "fp64" else 4
        return "mfma", N * 10.0 * F * F, N * (F * b + 6.0 * F * ab)
    if kernel == "bwd_heads":
        dims = [F] + list(hp.shared_dims) + list(hp.branch_dims)[:-1]
        n = N if head_entries is None else head_entries
        return "mfma", n * 2.0 * sum(2.0 * a * c for a, c in zip(dims[:-1], dims[1:])), N * F * b
    if kernel == "heads":
        dims = [F] + list(hp.shared_dims) + list(hp.branch_dims)
        n = N if head_entries is None else head_entries
        return "mfma", n * sum(2.0 * a * c for a, c in zip(dims[:-1], dims[1:])), N * F * b
    return None, 0.0, 0.0


def load_traffic(key: str, digest: str, kernel: str):
    """HBM bytes per launch of `kernel` in workload/precision `key`, from the
    stored counter measurement, or None when there is none for that kernel
    or the kernel sources changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = (json.load(f).get(key) or {}).get(kernel)
    except (OSError, ValueError, AttributeError):
        return None
    if not t or t.get("source_digest") != digest:
        return None
    return t.get("bytes_per_launch")


def cpu_baseline(name: str, batch, sample: int, blend_skip=None, forces=False):
    """Time the oracle (as it stands) on the first `sample` structures, one
    single-threaded worker per available core (blended heads when blend_skip
    is given; energies and forces when `forces`)."""
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    from concurrent.futures import ProcessPoolExecutor
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import helpers
    cores = len(os.sched_getaffinity(0))
    cores = min(cores, 16)
    idx = list(range(min(sample, batch.n_struct)))
    t0 = time.perf_counter()
    if forces:
        helpers.oracle_forces(name, batch, idx, workers=cores)
    else:
        helpers.oracle_energies(name, batch, idx, workers=cores, blend_skip=blend_skip)
    dt = time.perf_counter() - t0
    what = "FP64 NumPy PaiNN energies and reverse-pass forces" if forces else "FP64 NumPy PaiNN"
    return dict(value=len(idx) / dt, unit="structures/s", cores=cores, kind="oracle",
                sample=f"first {len(idx)} structures of the {name} batch, oracle (brute-force graph + "
                       f"{what}) in a pool of {cores} single-threaded processes, {dt:.1f} s wall")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="molecules_4096",
                    choices=["molecules_4096", "bulk_1024", "screening", "lead_model", "tiny_molecules"])
    ap.add_argument("--precision", default=None, choices=["fp64", "fp32", "bf16"])
    ap.add_argument("--blend", action="store_true",
                    help="blend every head with the model's branch-weighting MLP (screening model)")
    ap.add_argument("--skip", type=float, default=0.0,
                    help="with --blend: leave out heads whose weight is below this threshold")
    ap.add_argument("--forces", action="store_true",
                    help="energies and forces (painn_forces) instead of the energy forward")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="structures the CPU oracle baseline times (default 768; 256 with --forces)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="time without per-kernel events")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run one device-to-device copy of MIB MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (screening shards "
              "into independent batches per GPU, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    if args.copy_probe:
        n = args.copy_probe * (1 << 20) // 4
        x = torch.ones(n, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": 4 * n, "copy_probe_bytes_written": 4 * n}))
        return
    import synth
    from paper_2604_15380_amd import Runtime, painn_profile_enable, painn_profile_read

    name = args.workload
    spec = synth.WORKLOADS[name]
    prec = args.precision or spec["precision"]
    hp, W = synth.workload_weights(name)
    log(f"generating {name}")
    if spec.get("batch_atoms"):
        # a stream workload: its first batch (closed before 65,536 atoms)
        start, cnt = synth.screening_batches(3000, name=name)[0]
        batch = synth.make_batch(name, start, cnt)
    else:
        batch = synth.make_batch(name)
    rt = Runtime(0)
    model = rt.load_model(synth.weight_file_bytes(hp, W))
    inp = rt.upload_batch(batch)
    ds = inp["dataset_id"] if hp.n_heads > 1 else None
    graph = rt.build_graph(inp, hp.cutoff, max_neighbors=hp.max_neighbors)
    out = torch.empty(batch.n_struct, dtype=torch.float64, device=rt.device)

    if args.blend and hp.blend_dims is None:
        print(f"--blend needs a model with a branch-weighting MLP ({name} has none)", file=sys.stderr)
        sys.exit(2)
    if args.forces and prec == "bf16":
        print("--forces runs in FP64 or FP32", file=sys.stderr)
        sys.exit(2)
    fout = torch.empty((batch.n_atoms, 3), dtype=torch.float64, device=rt.device)

    def step():
        rt.build_graph(inp, hp.cutoff, graph=graph, max_neighbors=hp.max_neighbors)
        if args.forces and args.blend:
            rt.forces_blend(model, graph, prec, skip=args.skip, energies=out, forces=fout)
        elif args.forces:
            rt.forces(model, graph, prec, dataset_id=ds, energies=out, forces=fout)
        elif args.blend:
            rt.forward_blend(model, graph, prec, skip=args.skip, out=out)
        else:
            rt.forward(model, graph, prec, dataset_id=ds, out=out)

    log(f"{batch.n_struct} structures, {batch.n_atoms} atoms, {graph.n_edges} edges; warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    head_entries = None
    if args.blend:
        # (atom, head) entries the heads run: every kept head of each structure
        w = torch.empty((batch.n_struct, hp.n_heads), dtype=torch.float64, device=rt.device)
        rt.forward_blend(model, graph, prec, skip=args.skip, out=out, weights=w)
        kept = (w >= args.skip).sum(dim=1).cpu().numpy()
        head_entries = int(np.sum(np.diff(batch.struct_ptr) * kept))
        log(f"blended heads: {head_entries / max(1, batch.n_atoms):.2f} kept heads per atom")
        torch.cuda.synchronize()
    if not args.no_profile:
        painn_profile_read(rt.ctx)
        painn_profile_enable(rt.ctx, True)
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    T = time.perf_counter() - t0
    prof = {}
    if not args.no_profile:
        painn_profile_enable(rt.ctx, False)
        prof = painn_profile_read(rt.ctx)
    K = args.steps
    B, N, E = batch.n_struct, batch.n_atoms, graph.n_edges
    value = B * K / T
    log(f"{1e3 * T / K:.3f} ms/step, {value:.1f} structures/s")

    # PCIe-inclusive rate: pinned host inputs copied in, energies (and
    # forces) copied out
    host = {k: v.cpu().pin_memory() for k, v in inp.items() if torch.is_tensor(v)}
    out_h = torch.empty(B, dtype=torch.float64).pin_memory()
    fout_h = torch.empty((N, 3), dtype=torch.float64).pin_memory()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(K):
        for k, v in host.items():
            inp[k].copy_(v, non_blocking=True)
        step()
        out_h.copy_(out, non_blocking=True)
        if args.forces:
            fout_h.copy_(fout, non_blocking=True)
    torch.cuda.synchronize()
    T_pcie = time.perf_counter() - t1

    kernel_ms = {k: round(ms / K, 4) for k, (ms, n) in prof.items()}
    roofline = None
    if prof:
        cand = {k: v for k, v in prof.items() if kernel_work(k, hp, N, E, prec, head_entries)[0]}
        dom = max(cand, key=lambda k: cand[k][0])
        ms, launches = cand[dom]
        bound, flops, nbytes = kernel_work(dom, hp, N, E, prec, head_entries)
        avg_s = ms / launches / 1e3
        achieved = flops / avg_s / 1e12
        peak = PEAK[bound][prec]
        traffic = load_traffic(f"{name}/{prec}" + ("/forces" if args.forces else ""),
                               source_digest(args.forces), dom)
        roofline = dict(kernel=dom, bound=bound, achieved=round(achieved, 3), peak=peak, unit="TFLOP/s",
                        frac=round(achieved / peak, 4), traffic=traffic,
                        avg_launch_ms=round(avg_s * 1e3, 4), launches=launches,
                        algorithmic_flops_per_launch=flops, algorithmic_hbm_bytes_per_launch=nbytes,
                        achieved_hbm_GBps_algorithmic=round(nbytes / avg_s / 1e9, 1))

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline")
        sample = args.cpu_sample or (256 if args.forces else 768)
        cpu = cpu_baseline(name, batch, sample, args.skip if args.blend else None, forces=args.forces)

    res = {
        "metric": METRIC_FORCES if args.forces else METRIC, "value": round(value, 2), "unit": "structures/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": round(1e3 * T / K, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": DTYPE[prec], "data": "synthetic",
        "config": {"workload": name, "n_struct": B, "n_atoms": N, "n_edges": E, "F": hp.F,
                   "layers": hp.L, "rbf": hp.K, "rbf_type": ["gaussian", "bessel"][hp.rbf_type],
                   "cutoff": hp.cutoff, "max_neighbors": hp.max_neighbors, "heads": hp.n_heads,
                   "precision": prec, "forces": bool(args.forces),
                   "head_mode": (f"blended, skip < {args.skip:g}" if args.blend else
                                 ("dataset id" if hp.n_heads > 1 else "single"))},
        "edges_per_s": round(E * K / T, 1),
        "edge_messages_per_s": round(E * hp.L * K / T, 1),
        "pcie_inclusive_structures_per_s": round(B * K / T_pcie, 2),
        "kernel_ms_per_step": kernel_ms,
        "heads_per_atom": None if head_entries is None else round(head_entries / max(1, N), 3),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)
    graph.free()
    model.free()
    rt.close()


if __name__ == "__main__":
    main()
