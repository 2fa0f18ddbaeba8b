"""Benchmark of the batched PaiNN screening forward pass on one MI355X.

A step is one pass of the whole hot path over one batch already resident in
HBM: radius graph (painn_build_graph) + forward (embedding, L interaction
layers, heads, per-structure energies).  Default workload: 1024 periodic
cubic cells of 32-256 atoms (0.08 atoms/A^3, 85 elements, r_c = 6 A), F = 256,
6 layers, 32 Gaussian RBF, FP64 end to end -- the largest single-GPU batch.

--stream N walks N distinct consecutive batches of the screening stream
(each closed before 65,536 atoms) instead of repeating one batch: all N are
resident in HBM before the timed region; a second figure copies each next
batch host-to-device on a second stream while the current one runs.

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
# MI355X published peaks (dense), TFLOP/s: vector ALU (the BF16 mode's
# element-wise work runs in FP32) and matrix cores
PEAK = {
    "alu": {"fp64": 78.6, "fp32": 157.3, "bf16": 157.3},
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
    """Algorithmic work of ONE launch of a kernel class:
    (compute unit, flops on the matrix cores, flops on the vector ALU, HBM bytes).

    message: per edge 6KF (radial filter contraction over K basis functions
             for 3F channels, on the matrix cores) + 22F (cutoff and bias,
             scalar and vector messages, vector ALU); minimum HBM bytes: per
             atom h (3F), v in (3F), s (F) read and s (F), v out (3F) written,
             plus 8 bytes of CSR per edge.  The first layer's v is zero, so its
             launch forms 2 of the 3 filter parts (4KF), does half the
             elementwise work (11F) and reads no v; the figure per launch is the
             mean over the L launches.
    update:  per atom 22 F^2 (U/V 12F^2, gate MLP 10F^2) + 8 F^2 for the next
             layer's phi fused behind it (all but the last layer); minimum HBM
             bytes: s, v read (4F), s, v and the next h written (4F + 3F).
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
    ab = 8 if prec == "fp64" else 4
    if kernel == "message":
        filt = E * ((L - 1) * 6.0 * K * F + 4.0 * K * F) / L
        elem = E * ((L - 1) * 22.0 * F + 11.0 * F) / L
        nb = N * ((L - 1) * 11.0 + 8.0) / L * F * b + 8.0 * E
        return "alu", filt, elem, nb
    if kernel == "update":
        fl = N * (22.0 * F * F + 8.0 * F * F * (L - 1) / L)
        return "mfma", fl, 0.0, N * (8.0 * F + 3.0 * F * (L - 1) / L) * b
    if kernel == "phi":
        return "mfma", N * 8.0 * F * F, 0.0, N * 4.0 * F * b
    if kernel == "bwd_message":
        return "alu", E * 12.0 * K * F, E * 36.0 * F, N * (6.0 * F * b + 10.0 * F * ab) + 8.0 * E
    if kernel == "bwd_update":
        return "mfma", N * 22.0 * F * F, 0.0, N * (9.0 * F * b + 8.0 * F * ab)
    if kernel == "bwd_phi":
        return "mfma", N * 10.0 * F * F, 0.0, N * (F * b + 6.0 * F * ab)
    if kernel == "bwd_heads":
        dims = [F] + list(hp.shared_dims) + list(hp.branch_dims)[:-1]
        n = N if head_entries is None else head_entries
        return "mfma", n * 2.0 * sum(2.0 * a * c for a, c in zip(dims[:-1], dims[1:])), 0.0, N * F * b
    if kernel == "heads":
        dims = [F] + list(hp.shared_dims) + list(hp.branch_dims)
        n = N if head_entries is None else head_entries
        return "mfma", n * sum(2.0 * a * c for a, c in zip(dims[:-1], dims[1:])), 0.0, N * F * b
    return None, 0.0, 0.0, 0.0


def roofline_entry(kernel: str, prec: str, mfma_flops: float, valu_flops: float, nbytes: float,
                   unit_kind: str, ms: float, launches: int, traffic):
    """Roofline of one kernel class from its algorithmic work per launch and
    its measured mean launch time.  The binding roof is the larger of the
    ideal compute time (matrix-core flops at the precision's MFMA peak plus
    vector flops at the vector peak) and the ideal HBM time (algorithmic
    bytes at 8 TB/s); `frac` is achieved / peak on that roof."""
    avg_s = ms / launches / 1e3
    t_comp = (mfma_flops / (PEAK["mfma"][prec] * 1e12) + valu_flops / (PEAK["alu"][prec] * 1e12))
    t_mem = nbytes / (HBM_PEAK_GBS * 1e9)
    flops = mfma_flops + valu_flops
    gbs = nbytes / avg_s / 1e9
    tflops = flops / avg_s / 1e12
    if t_mem > t_comp:
        bound, achieved, peak, unit = "hbm", gbs, HBM_PEAK_GBS, "GB/s"
    else:
        # the compute roof of a launch that mixes units: its flops over the
        # ideal compute time (equal to the published peak when one unit runs
        # all of it, or both units share a peak as in FP32 and FP64)
        bound, achieved, unit = unit_kind, tflops, "TFLOP/s"
        peak = flops / t_comp / 1e12 if t_comp > 0 else PEAK[unit_kind][prec]
    return dict(kernel=kernel, bound=bound, achieved=round(achieved, 3), peak=round(peak, 2), unit=unit,
                frac=round(achieved / peak, 4), traffic=traffic, avg_launch_ms=round(avg_s * 1e3, 4),
                launches=launches, algorithmic_flops_per_launch=flops,
                algorithmic_hbm_bytes_per_launch=nbytes, achieved_TFLOPs=round(tflops, 3),
                achieved_hbm_GBps_algorithmic=round(gbs, 1),
                compute_frac=round(t_comp / avg_s, 4), hbm_frac=round(t_mem / avg_s, 4),
                traffic_over_algorithmic=None if traffic is None else round(traffic / nbytes, 3))


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


# Worker processes of the CPU baseline: one single-threaded oracle process per
# core of the host's share, at most this many (a one-GPU share of the GPU
# hosts is 16 cores; the machines expose more than a job may use).
CPU_SHARE = 16


def blas_name() -> str:
    try:
        from threadpoolctl import threadpool_info
        info = [d for d in threadpool_info() if d.get("user_api") == "blas"]
        if info:
            return f"{info[0].get('internal_api')} {info[0].get('version') or ''}".strip()
    except Exception:
        pass
    return "unknown"


def cpu_baseline(name: str, batch, sample: int, blend_skip=None, forces=False):
    """Time the oracle (as it stands) on the first `sample` structures, one
    single-threaded worker per core of the host share (blended heads when
    blend_skip is given; energies and forces when `forces`)."""
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import helpers
    affinity = len(os.sched_getaffinity(0))
    idx = list(range(min(sample, batch.n_struct)))
    cores = max(1, min(affinity, CPU_SHARE, len(idx)))
    t0 = time.perf_counter()
    if forces:
        helpers.oracle_forces(name, batch, idx, workers=cores)
    else:
        helpers.oracle_energies(name, batch, idx, workers=cores, blend_skip=blend_skip)
    dt = time.perf_counter() - t0
    what = "FP64 NumPy PaiNN energies and reverse-pass forces" if forces else "FP64 NumPy PaiNN"
    return dict(value=len(idx) / dt, unit="structures/s", cores=cores, kind="oracle",
                sample=f"first {len(idx)} structures of the {name} batch, oracle (brute-force graph + "
                       f"{what}) in a pool of {cores} single-threaded processes, {dt:.1f} s wall",
                os_cpu_count=os.cpu_count(), affinity_cores=affinity, worker_cap=CPU_SHARE,
                blas=blas_name(), wall_s=round(dt, 2))


def _gen_batch(args):
    name, start, cnt = args
    import synth
    return synth.make_batch(name, start, cnt)


def stream_batches(name: str, n: int):
    """The first n batches of a stream workload, generated in a process pool."""
    import synth
    from concurrent.futures import ProcessPoolExecutor
    spec = synth.WORKLOADS[name]
    per = max(1, spec["batch_atoms"] // 40)
    ranges = synth.screening_batches(per * (n + 1), name=name)[:n]
    if len(ranges) < n:
        raise SystemExit(f"only {len(ranges)} batches generated")
    workers = max(1, min(CPU_SHARE, len(os.sched_getaffinity(0)), n))
    with ProcessPoolExecutor(workers) as ex:
        return list(ex.map(_gen_batch, [(name, s, c) for s, c in ranges]))


METRIC_TRAIN = "PaiNN FP64 training structures/s on 1 MI355X (energy+force MAE loss, AdamW)"


def adamw_bytes(n_params: int) -> float:
    """HBM bytes of one AdamW update: weights, both moments read and written,
    the gradient read (8-byte values)."""
    return n_params * 8.0 * 7


def bench_train(args):
    """Training steps of the lead model's shape (Table 5: batch of 25
    structures per GPU, MAE on energies and forces with force weight 94.8,
    AdamW at 6.34e-4, FP64): each step builds the capped graph of the next 25
    structures of the stream and runs painn_trainer_step on synthetic
    reference energies and forces."""
    import numpy as np
    import torch
    import synth
    from paper_2604_15380_amd import Runtime, painn_profile_enable, painn_profile_read
    from paper_2604_15380_amd import binding as Bd
    name = "lead_model"
    per = 25
    hp, W = synth.workload_weights(name)
    hp.blend_dims = None
    W = {k: v for k, v in W.items() if not k.startswith("blend")}
    K, Wu = args.steps, args.warmup
    log(f"generating {K + Wu} batches of {per} {name} structures")
    rng = np.random.default_rng(7)
    batches = [synth.make_batch(name, per * k, per) for k in range(K + Wu)]
    refs = [(rng.standard_normal(b.n_struct) * 2.0, rng.standard_normal((b.n_atoms, 3)) * 0.5) for b in batches]
    rt = Runtime(0)
    model = rt.load_model(synth.weight_file_bytes(hp, W))
    tr = Bd.painn_trainer_create(rt.ctx, model.handle, None)
    n_params = Bd.painn_trainer_params(rt.ctx, tr)
    inputs = [rt.upload_batch(b) for b in batches]
    er = [torch.as_tensor(e, device=rt.device) for e, _ in refs]
    fr = [torch.as_tensor(np.ascontiguousarray(f), device=rt.device) for _, f in refs]
    loss = torch.zeros(3, dtype=torch.float64, device=rt.device)
    graph = rt.build_graph(inputs[0], hp.cutoff, max_neighbors=hp.max_neighbors)
    edges = []

    def step(k):
        inp = inputs[k]
        rt.build_graph(inp, hp.cutoff, graph=graph, max_neighbors=hp.max_neighbors)
        Bd.painn_trainer_step(rt.ctx, tr, graph.handle, inp["dataset_id"].data_ptr(), er[k].data_ptr(),
                              fr[k].data_ptr(), loss.data_ptr())
        return graph.n_edges

    for k in range(Wu):
        step(K + k)
    torch.cuda.synchronize()
    painn_profile_read(rt.ctx)
    painn_profile_enable(rt.ctx, True)
    log(f"timing {K} training steps")
    t0 = time.perf_counter()
    for k in range(K):
        edges.append(step(k))
    torch.cuda.synchronize()
    T = time.perf_counter() - t0
    painn_profile_enable(rt.ctx, False)
    prof = painn_profile_read(rt.ctx)
    last_loss = loss.cpu().numpy().tolist()
    tot_B = sum(batches[k].n_struct for k in range(K))
    tot_N = sum(batches[k].n_atoms for k in range(K))
    value = tot_B / T
    log(f"{1e3 * T / K:.3f} ms/step, {value:.1f} structures/s, last loss {last_loss}")
    kernel_ms = {k: round(ms / K, 4) for k, (ms, n) in prof.items()}
    roofline = None
    if "train_adamw" in prof:
        ms, n = prof["train_adamw"]
        avg = ms / n / 1e3
        nb = adamw_bytes(n_params)
        roofline = dict(kernel="train_adamw", bound="hbm", achieved=round(nb / avg / 1e9, 1), peak=HBM_PEAK_GBS,
                        unit="GB/s", frac=round(nb / avg / 1e9 / HBM_PEAK_GBS, 4), traffic=None,
                        avg_launch_ms=round(avg * 1e3, 4), launches=n, algorithmic_hbm_bytes_per_launch=nb,
                        note="the optimizer update; the gradient passes are FP64 vector-ALU kernels "
                             "without an algorithmic flop count")
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline (one training-step gradient)")
        os.environ.setdefault("OMP_NUM_THREADS", "1")
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        import helpers
        affinity = len(os.sched_getaffinity(0))
        workers = max(1, min(affinity, CPU_SHARE, per))
        b = batches[0]
        t1 = time.perf_counter()
        helpers.oracle_train_grad(hp, name, b, refs[0][0], refs[0][1], 94.8, workers=workers)
        dt = time.perf_counter() - t1
        cpu = dict(value=b.n_struct / dt, unit="structures/s", cores=workers, kind="oracle",
                   sample=f"one training-step gradient of the first {b.n_struct}-structure batch ({b.n_atoms} "
                          f"atoms): oracle forces, then the complex-step loss gradient, in a pool of {workers} "
                          f"single-threaded processes, {dt:.1f} s wall",
                   os_cpu_count=os.cpu_count(), affinity_cores=affinity, worker_cap=CPU_SHARE,
                   blas=blas_name(), wall_s=round(dt, 2))
    res = {
        "metric": METRIC_TRAIN, "value": round(value, 2), "unit": "structures/s", "n_gpus": 1, "steps": K,
        "warmup": Wu, "ms_per_step": round(1e3 * T / K, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{name} training, {per} structures per step, {K} distinct batches",
                   "n_struct": tot_B, "n_atoms": tot_N, "n_edges": int(sum(edges)), "F": hp.F, "layers": hp.L,
                   "rbf": hp.K, "rbf_type": "bessel", "cutoff": hp.cutoff, "max_neighbors": hp.max_neighbors,
                   "heads": hp.n_heads, "precision": "fp64", "loss": "MAE(E) + 94.8 MAE(F)",
                   "optimizer": "AdamW lr 6.34e-4, betas (0.9, 0.999), eps 1e-8, weight decay 0.01",
                   "n_params": n_params,
                   "weights": f"random, dense ~ N(0, 1/fan_in), radial filter x {synth.FILTER_GAIN:g}"},
        "kernel_ms_per_step": kernel_ms,
        "last_loss": last_loss,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)
    Bd.painn_trainer_free(tr)
    graph.free()
    model.free()
    rt.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="bulk_1024",
                    choices=["molecules_4096", "bulk_1024", "screening", "lead_model", "tiny_molecules"])
    ap.add_argument("--precision", default=None, choices=["fp64", "fp32", "bf16"])
    ap.add_argument("--stream", type=int, default=0, metavar="N",
                    help="time N distinct consecutive batches of a stream workload (screening, "
                         "lead_model) instead of repeating its first batch")
    ap.add_argument("--blend", action="store_true",
                    help="blend every head with the model's branch-weighting MLP (screening model)")
    ap.add_argument("--skip", type=float, default=0.0,
                    help="with --blend: leave out heads whose weight is below this threshold")
    ap.add_argument("--forces", action="store_true",
                    help="energies and forces (painn_forces) instead of the energy forward")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="structures the CPU oracle baseline times (default: 16 for bulk_1024, 256 with "
                         "--forces, else 768)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="time without per-kernel events")
    ap.add_argument("--train", action="store_true",
                    help="time training steps (lead model shape, 25 structures per step, FP64)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run one device-to-device copy of MIB MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (screening shards "
              "into independent batches per GPU, see the design notes)", file=sys.stderr)
        sys.exit(2)

    if args.train:
        bench_train(args)
        return
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
    if args.stream and name not in ("screening", "lead_model"):
        name = "screening"
    spec = synth.WORKLOADS[name]
    prec = args.precision or spec["precision"]
    hp, W = synth.workload_weights(name)
    if args.blend and hp.blend_dims is None:
        print(f"--blend needs a model with a branch-weighting MLP ({name} has none)", file=sys.stderr)
        sys.exit(2)
    if args.forces and prec == "bf16":
        print("--forces runs in FP64 or FP32", file=sys.stderr)
        sys.exit(2)
    log(f"generating {name}" + (f", {args.stream} stream batches" if args.stream else ""))
    if args.stream:
        batches = stream_batches(name, args.stream)
    elif spec.get("batch_atoms"):
        # a stream workload: its first batch (closed before 65,536 atoms)
        start, cnt = synth.screening_batches(3000, name=name)[0]
        batches = [synth.make_batch(name, start, cnt)]
    else:
        batches = [synth.make_batch(name)]
    rt = Runtime(0)
    model = rt.load_model(synth.weight_file_bytes(hp, W))
    inputs = [rt.upload_batch(b) for b in batches]
    graph = rt.build_graph(inputs[0], hp.cutoff, max_neighbors=hp.max_neighbors)
    Bmax = max(b.n_struct for b in batches)
    Nmax = max(b.n_atoms for b in batches)
    outs = [torch.empty(b.n_struct, dtype=torch.float64, device=rt.device) for b in batches]
    fout = torch.empty((Nmax, 3), dtype=torch.float64, device=rt.device)

    def step(k):
        inp = inputs[k]
        rt.build_graph(inp, hp.cutoff, graph=graph, max_neighbors=hp.max_neighbors)
        ds = inp["dataset_id"] if hp.n_heads > 1 else None
        out = outs[k]
        if args.forces and args.blend:
            rt.forces_blend(model, graph, prec, skip=args.skip, energies=out, forces=fout)
        elif args.forces:
            rt.forces(model, graph, prec, dataset_id=ds, energies=out, forces=fout)
        elif args.blend:
            rt.forward_blend(model, graph, prec, skip=args.skip, out=out)
        else:
            rt.forward(model, graph, prec, dataset_id=ds, out=out)
        return graph.n_edges

    # the batches a timed pass walks: every stream batch once, or the one
    # batch K times
    K = args.stream if args.stream else args.steps
    order = list(range(len(batches))) if args.stream else [0] * K
    tot_B = sum(batches[k].n_struct for k in order)
    tot_N = sum(batches[k].n_atoms for k in order)
    log(f"{len(batches)} batch(es): {batches[0].n_struct} structures, {batches[0].n_atoms} atoms, "
        f"{graph.n_edges} edges in the first; warmup {args.warmup}")
    for w in range(args.warmup):
        step(order[w % len(order)])
    torch.cuda.synchronize()
    head_entries = None
    if args.blend:
        # (atom, head) entries the heads run: every kept head of each structure
        b0 = batches[order[0]]
        rt.build_graph(inputs[order[0]], hp.cutoff, graph=graph, max_neighbors=hp.max_neighbors)
        w = torch.empty((b0.n_struct, hp.n_heads), dtype=torch.float64, device=rt.device)
        rt.forward_blend(model, graph, prec, skip=args.skip, out=outs[order[0]], weights=w)
        kept = (w >= args.skip).sum(dim=1).cpu().numpy()
        head_entries = int(np.sum(np.diff(b0.struct_ptr) * kept))
        log(f"blended heads: {head_entries / max(1, b0.n_atoms):.2f} kept heads per atom")
        torch.cuda.synchronize()
    if not args.no_profile:
        painn_profile_read(rt.ctx)
        painn_profile_enable(rt.ctx, True)
    log(f"timing {K} steps")
    edges = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in order:
        edges.append(step(k))
    torch.cuda.synchronize()
    T = time.perf_counter() - t0
    prof = {}
    if not args.no_profile:
        painn_profile_enable(rt.ctx, False)
        prof = painn_profile_read(rt.ctx)
    tot_E = sum(edges)
    value = tot_B / T
    log(f"{1e3 * T / K:.3f} ms/step, {value:.1f} structures/s")

    # PCIe-inclusive rate: pinned host inputs copied in, energies (and
    # forces) copied out.  Repeated batch: in the step's own stream order.
    # Stream: the next batch's inputs go up on a second stream while the
    # current batch runs (two device buffer sets).
    keys = ["struct_ptr", "pos", "species", "cell", "pbc", "dataset_id"]
    host = [{k: v.cpu().pin_memory() for k, v in inp.items() if k in keys} for inp in inputs]
    out_h = torch.empty(Bmax, dtype=torch.float64).pin_memory()
    fout_h = torch.empty((Nmax, 3), dtype=torch.float64).pin_memory()
    cur = torch.cuda.current_stream()
    if args.stream:
        copy_s = torch.cuda.Stream(device=rt.device)
        sets = [{k: inputs[0][k].new_empty(max(h[k].shape[0] for h in host), *inputs[0][k].shape[1:])
                 for k in keys} for _ in range(2)]
        up_ev = [torch.cuda.Event() for _ in range(2)]
        done_ev = [torch.cuda.Event() for _ in range(2)]

        def upload(k):
            slot = k % 2
            with torch.cuda.stream(copy_s):
                copy_s.wait_event(done_ev[slot])
                view = {}
                for key in keys:
                    n = host[k][key].shape[0]
                    sets[slot][key][:n].copy_(host[k][key], non_blocking=True)
                    view[key] = sets[slot][key][:n]
                up_ev[slot].record(copy_s)
            view.update(n_struct=inputs[k]["n_struct"], n_atoms=inputs[k]["n_atoms"],
                        any_pbc=inputs[k]["any_pbc"])
            return view

        for ev in done_ev:
            ev.record(cur)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        staged = upload(order[0])
        for i, k in enumerate(order):
            cur.wait_event(up_ev[k % 2])
            now = staged
            if i + 1 < len(order):
                staged = upload(order[i + 1])
            saved = inputs[k]
            inputs[k] = now
            step(k)
            inputs[k] = saved
            done_ev[k % 2].record(cur)
            out_h[:batches[k].n_struct].copy_(outs[k], non_blocking=True)
            if args.forces:
                fout_h[:batches[k].n_atoms].copy_(fout[:batches[k].n_atoms], non_blocking=True)
        torch.cuda.synchronize()
        T_pcie = time.perf_counter() - t1
    else:
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for k in order:
            for key, v in host[k].items():
                inputs[k][key].copy_(v, non_blocking=True)
            step(k)
            out_h[:batches[k].n_struct].copy_(outs[k], non_blocking=True)
            if args.forces:
                fout_h[:batches[k].n_atoms].copy_(fout[:batches[k].n_atoms], non_blocking=True)
        torch.cuda.synchronize()
        T_pcie = time.perf_counter() - t1

    kernel_ms = {k: round(ms / K, 4) for k, (ms, n) in prof.items()}
    roofline, kernels = None, {}
    if prof:
        key = f"{name}/{prec}" + ("/forces" if args.forces else "")
        digest = source_digest(args.forces)
        for kern, (ms, launches) in prof.items():
            # work summed over the batches the timed pass walked, per launch
            works = [kernel_work(kern, hp, batches[k].n_atoms, e, prec, head_entries)
                     for k, e in zip(order, edges)]
            if not works[0][0]:
                continue
            # per launch: the mean over the walked batches (each batch runs
            # the same launches of every class)
            mf = sum(w[1] for w in works) / K
            vf = sum(w[2] for w in works) / K
            nb = sum(w[3] for w in works) / K
            kernels[kern] = roofline_entry(kern, prec, mf, vf, nb, works[0][0], ms, launches,
                                           None if args.stream else load_traffic(key, digest, kern))
        if kernels:
            dom = max(kernels, key=lambda k: prof[k][0])
            roofline = dict(kernels[dom])
            roofline["kernels"] = {k: {x: v[x] for x in ("bound", "achieved", "peak", "unit", "frac", "traffic",
                                                         "avg_launch_ms", "compute_frac", "hbm_frac",
                                                         "achieved_hbm_GBps_algorithmic")}
                                   for k, v in kernels.items() if k != dom}

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle baseline")
        sample = args.cpu_sample or (256 if args.forces else 16 if name == "bulk_1024" else 768)
        cpu = cpu_baseline(name, batches[0], sample, args.skip if args.blend else None, forces=args.forces)

    res = {
        "metric": METRIC_FORCES if args.forces else METRIC, "value": round(value, 2), "unit": "structures/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": round(1e3 * T / K, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": DTYPE[prec], "data": "synthetic",
        "config": {"workload": name + (f" stream, {K} distinct batches" if args.stream else ""),
                   "n_struct": tot_B // K if not args.stream else tot_B,
                   "n_atoms": tot_N // K if not args.stream else tot_N,
                   "n_edges": tot_E // K if not args.stream else tot_E, "F": hp.F,
                   "layers": hp.L, "rbf": hp.K, "rbf_type": ["gaussian", "bessel"][hp.rbf_type],
                   "cutoff": hp.cutoff, "max_neighbors": hp.max_neighbors, "heads": hp.n_heads,
                   "precision": prec, "forces": bool(args.forces),
                   "head_mode": (f"blended, skip < {args.skip:g}" if args.blend else
                                 ("dataset id" if hp.n_heads > 1 else "single")),
                   "weights": f"random, dense ~ N(0, 1/fan_in), radial filter x {synth.FILTER_GAIN:g}"},
        "edges_per_s": round(tot_E / T, 1),
        "edge_messages_per_s": round(tot_E * hp.L / T, 1),
        ("pcie_overlapped_structures_per_s" if args.stream else "pcie_inclusive_structures_per_s"):
            round(tot_B / T_pcie, 2),
        "kernel_ms_per_step": kernel_ms,
        "heads_per_atom": None if head_entries is None else round(head_entries / max(1, batches[0].n_atoms), 3),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)
    graph.free()
    model.free()
    rt.close()


if __name__ == "__main__":
    main()
