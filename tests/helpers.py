"""Shared test helpers: GPU runtime fixture, parallel oracle evaluation and
the energy tolerance metric."""
from __future__ import annotations

import os
from concurrent.futures import ProcessPoolExecutor

import numpy as np

import synth

# Energy acceptance: |E - E_ref| <= tol * sum_i |e_i^ref| per structure (the
# error bound of a floating-point sum of per-atom energies; plain |E_ref| is
# reported beside it).  Tolerances per precision:
TOL = {"fp64": 1e-10, "fp32": 1e-5, "bf16": 2e-2}


def bf16_round(x):
    """Round FP64 values to the nearest bfloat16 value (8 significant bits),
    ties to even, in one step from FP64 (reading R14)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def stored_weights(W: dict, precision: str) -> dict:
    """The weights a precision mode computes with: BF16 mode stores every
    weight in BF16 (R13, R14), so its FP64 reference is the oracle run on the
    BF16-rounded weights (the rounding alone moves some small structures'
    energies by more than the BF16 tolerance: R29).  Other modes: W."""
    if precision != "bf16":
        return W
    return {k: bf16_round(v) for k, v in W.items()}


def _single_thread_blas():
    """Pool initializer: one BLAS thread per worker process (the pool itself
    provides the parallelism; inherited thread counts would oversubscribe)."""
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except ImportError:
        pass


def _oracle_job(args):
    from oracle.painn import structure_forward, structure_forward_blend
    name, batch_tuple, idx, blend_skip, stored = args
    hp, W = synth.workload_weights(name)
    W = stored_weights(W, stored)
    out = []
    for k, (pos, z, cell, pbc, ds) in zip(idx, batch_tuple):
        if blend_skip is None:
            o = structure_forward(pos, z, cell, pbc, ds if hp.n_heads > 1 else 0, hp, W)
        else:
            o = structure_forward_blend(pos, z, cell, pbc, hp, W, skip=blend_skip)
        out.append((k, o["E"], float(np.sum(np.abs(o["e"])))))
    return out


def _oracle_forces_job(args):
    from oracle.forces import structure_forces, structure_forces_blend
    name, batch_tuple, idx, blend_skip = args
    hp, W = synth.workload_weights(name)
    if blend_skip is not None:
        return [(k, structure_forces_blend(pos, z, cell, pbc, hp, W, skip=blend_skip))
                for k, (pos, z, cell, pbc, ds) in zip(idx, batch_tuple)]
    return [(k, structure_forces(pos, z, cell, pbc, ds if hp.n_heads > 1 else 0, hp, W)["F"])
            for k, (pos, z, cell, pbc, ds) in zip(idx, batch_tuple)]


def oracle_forces(name: str, batch, idx, workers: int | None = None, blend_skip=None):
    """Oracle forces of structures `idx` of `batch` (list of [n_b, 3]), in a
    process pool; blend_skip given: the oracle's blended-heads result dicts
    (F, w, ...) with heads below blend_skip left out."""
    idx = [int(i) for i in idx]
    workers = workers or min(16, os.cpu_count() or 1, max(1, len(idx)))
    chunks = [idx[w::workers] for w in range(workers)]
    jobs = [(name, [batch.structure(k) for k in c], c, blend_skip) for c in chunks if c]
    res = {}
    with ProcessPoolExecutor(workers, initializer=_single_thread_blas) as ex:
        for part in ex.map(_oracle_forces_job, jobs):
            res.update(dict(part))
    return [res[k] for k in idx]


def oracle_energies(name: str, batch, idx, workers: int | None = None, blend_skip=None, stored: str = "fp64"):
    """Oracle (E, sum|e|) of structures `idx` of `batch`, in a process pool;
    blend_skip given: every head blended, heads below it left out; stored =
    "bf16": on the BF16-rounded weights (`stored_weights`)."""
    idx = [int(i) for i in idx]
    workers = workers or min(16, os.cpu_count() or 1, max(1, len(idx)))
    chunks = [idx[w::workers] for w in range(workers)]
    jobs = [(name, [batch.structure(k) for k in c], c, blend_skip, stored) for c in chunks if c]
    res = {}
    if workers == 1:
        for j in jobs:
            for k, e, a in _oracle_job(j):
                res[k] = (e, a)
    else:
        with ProcessPoolExecutor(workers, initializer=_single_thread_blas) as ex:
            for part in ex.map(_oracle_job, jobs):
                for k, e, a in part:
                    res[k] = (e, a)
    E = np.array([res[k][0] for k in idx])
    A = np.array([res[k][1] for k in idx])
    return E, A


def _oracle_blend_job(args):
    from oracle.painn import structure_forward_blend
    name, batch_tuple, idx, skip, stored = args
    hp, W = synth.workload_weights(name)
    W = stored_weights(W, stored)
    return [(k, structure_forward_blend(pos, z, cell, pbc, hp, W, skip=skip))
            for k, (pos, z, cell, pbc, ds) in zip(idx, batch_tuple)]


def oracle_blend(name: str, batch, idx, skip: float, workers: int | None = None, stored: str = "fp64"):
    """The oracle's blended-heads results (dicts with E, e, w, E_heads) of
    structures `idx` of `batch`, in a process pool (stored as in
    `oracle_energies`)."""
    idx = [int(i) for i in idx]
    workers = workers or min(16, os.cpu_count() or 1, max(1, len(idx)))
    chunks = [idx[w::workers] for w in range(workers)]
    jobs = [(name, [batch.structure(k) for k in c], c, skip, stored) for c in chunks if c]
    res = {}
    with ProcessPoolExecutor(workers, initializer=_single_thread_blas) as ex:
        for part in ex.map(_oracle_blend_job, jobs):
            res.update(dict(part))
    return [res[k] for k in idx]


def check_energies(E_gpu, E_ref, A_ref, tol: float, label: str = ""):
    """Assert the tolerance on |E - E_ref| / sum_i |e_i^ref| per structure and
    report the plain relative error |E - E_ref| / |E_ref| beside it: its
    maximum and the share of structures within `tol` by that measure (it
    is ill-conditioned where E nearly cancels over the atoms).  Prints one
    line; returns (max normalised error, max plain relative error)."""
    E_gpu = np.asarray(E_gpu, dtype=np.float64)
    err = np.abs(E_gpu - E_ref)
    norm = err / A_ref
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.where(E_ref != 0, err / np.abs(E_ref), np.where(err == 0, 0.0, np.inf))
    worst = int(np.argmax(norm))
    share = float(np.mean(rel <= tol)) if len(rel) else 1.0
    print(f"{label}: {len(E_gpu)} structures; max |dE|/sum|e| = {norm.max() if len(norm) else 0.0:.3e}; "
          f"max |dE|/|E| = {rel.max() if len(rel) else 0.0:.3e}; "
          f"{100 * share:.2f}% within {tol:.0e} plain relative", flush=True)
    assert np.all(np.isfinite(E_gpu)), f"{label}: non-finite energies"
    assert norm.max() <= tol, (f"{label}: max |dE|/sum|e| = {norm.max():.3e} > {tol:.1e} "
                               f"at sample {worst} (E={E_gpu[worst]!r}, ref={E_ref[worst]!r})")
    return float(norm.max()), float(rel.max())


def report_vs_master(E_gpu, E_master, A_master, E_stored, tol: float, label: str = ""):
    """Accuracy against the oracle on the FP64 master weights, reported (not
    asserted) beside a BF16 parity check made against the oracle on the
    BF16-rounded weights: the worst |dE| / sum|e|, the share of structures
    within tol, and how far the weight rounding alone moves E."""
    E_gpu = np.asarray(E_gpu, dtype=np.float64)
    err = np.abs(E_gpu - E_master) / A_master
    wq = np.abs(np.asarray(E_stored) - E_master) / A_master
    print(f"{label} vs the FP64-weight oracle: max |dE|/sum|e| = {err.max():.3e}, "
          f"{100 * np.mean(err <= tol):.2f}% within {tol:.0e}; weight rounding alone: max {wq.max():.3e}",
          flush=True)
    return float(err.max())


def check_workload_energies(E_gpu, name: str, batch, idx, precision: str, label: str, workers=None):
    """Parity of GPU energies of structures idx of a workload batch with the
    FP64 oracle on the weights the precision mode stores (R29), at the
    precision's tolerance; in BF16 also the report against the master
    weights.  Returns (max normalised error, max plain relative error)."""
    Er, Ar = oracle_energies(name, batch, idx, workers, stored=precision)
    out = check_energies(E_gpu, Er, Ar, TOL[precision], label)
    if precision == "bf16":
        Em, Am = oracle_energies(name, batch, idx, workers)
        report_vs_master(E_gpu, Em, Am, Er, TOL[precision], label)
    return out


def check_forces(Fg, batch, ref_F, idx, tol: float, label: str = ""):
    """Per structure k of idx: max |F - F_ref| over its atoms and components
    <= tol * max |F_ref| of the structure (a structure with no force must get
    exactly zero).  Returns the worst ratio."""
    worst = 0.0
    for k, Fr in zip(idx, ref_F):
        lo, hi = int(batch.struct_ptr[k]), int(batch.struct_ptr[k + 1])
        Fk = np.asarray(Fg[lo:hi])
        assert np.all(np.isfinite(Fk)), f"{label}: non-finite forces in structure {k}"
        scale = float(np.abs(Fr).max()) if hi > lo else 0.0
        err = float(np.abs(Fk - Fr).max()) if hi > lo else 0.0
        if scale == 0.0:
            assert err == 0.0, f"{label}: structure {k} has no force but got {err:.3e}"
            continue
        worst = max(worst, err / scale)
        assert err <= tol * scale, f"{label}: structure {k}: max|dF| = {err:.3e} > {tol:.0e} * {scale:.3e}"
    print(f"{label}: {len(idx)} structures; worst max|dF|/max|F| = {worst:.3e}", flush=True)
    return worst


# Blended heads: absolute tolerance on the head weights (in [0, 1]) and the
# relative band around the skip threshold inside which the two sides may
# decide a head differently (the weights carry the precision's rounding)
W_TOL = {"fp64": 1e-12, "fp32": 1e-5, "bf16": 5e-3}


def check_blend(E, w_gpu, refs, idx, skip: float, precision: str, label: str = ""):
    """Blended energies of structures idx against the oracle's results
    `refs` (dicts with E, e, w, E_heads): weights within W_TOL, every head
    outside the undecided band kept or skipped alike, and the energy within
    the precision's tolerance of sum_i |e_i| after adding the contribution of
    undecided heads (those whose reference weight lies within W_TOL of the
    threshold) to the allowed error.  Returns the worst normalised error."""
    worst = 0.0
    n_heads = len(refs[0]["w"]) if refs else 0
    for k, o in zip(idx, refs):
        assert np.abs(w_gpu[k] - o["w"]).max() <= W_TOL[precision], (label, k)
        undecided = (np.abs(o["w"] - skip) <= W_TOL[precision]) if skip > 0 \
            else np.zeros(n_heads, bool)
        assert np.array_equal((w_gpu[k] >= skip)[~undecided], (o["w"] >= skip)[~undecided]), (label, k)
        slack = 1.1 * float(np.sum((o["w"][undecided] + W_TOL[precision]) * np.abs(o["E_heads"][undecided])))
        err = (abs(E[k] - o["E"]) - slack) / max(np.abs(o["e"]).sum(), 1e-300)
        worst = max(worst, err)
    print(f"{label}: {len(idx)} structures; worst blended |dE|/sum|e| = {worst:.3e}", flush=True)
    assert worst <= TOL[precision], (label, worst)
    return worst


def _oracle_train_job(args):
    from oracle.forces import structure_forces
    from oracle.train import structure_loss_grad_terms
    hp, W, structs, idx, c, u, stage = args
    if isinstance(W, str):
        # a workload's weights, regenerated here instead of shipped to the
        # worker (the router's arrays play no part in training)
        _, W = synth.workload_weights(W)
        W = {k: v for k, v in W.items() if not k.startswith("blend")}
    out = []
    for k, (pos, z, cell, pbc, ds) in zip(idx, structs):
        di = int(ds) if hp.n_heads > 1 else 0
        if stage == "forces":
            o = structure_forces(pos, z, cell, pbc, di, hp, W)
            out.append((k, (o["E"], o["F"])))
        else:
            out.append((k, structure_loss_grad_terms(pos, z, cell, pbc, di, hp, W, c[k], u[k])))
    return out


def oracle_train_grad(hp, W, batch, E_ref, F_ref, force_weight: float, workers: int | None = None):
    """oracle.train.loss_and_grad evaluated structure by structure in a
    process pool and summed in structure order: dict(loss, loss_E, loss_F,
    E, F, grad).  W may be a workload name (its weights without the router)."""
    B, N = batch.n_struct, batch.n_atoms
    workers = workers or min(16, os.cpu_count() or 1, max(1, B))
    idx = list(range(B))
    chunks = [idx[w::workers] for w in range(workers)]

    def run(stage, c=None, u=None):
        jobs = [(hp, W, [batch.structure(k) for k in ch], ch, c, u, stage) for ch in chunks if ch]
        res = {}
        with ProcessPoolExecutor(len(jobs), initializer=_single_thread_blas) as ex:
            for part in ex.map(_oracle_train_job, jobs):
                res.update(dict(part))
        return res

    fo = run("forces")
    E = np.array([fo[k][0] for k in idx])
    Fo = np.concatenate([fo[k][1] for k in idx]) if N else np.zeros((0, 3))
    rE = E - np.asarray(E_ref, dtype=np.float64)
    rF = Fo - np.asarray(F_ref, dtype=np.float64).reshape(N, 3)
    c = {k: float(np.sign(rE[k]) / B) for k in idx}
    u_all = force_weight * np.sign(rF) / (3 * N)
    u = {k: u_all[int(batch.struct_ptr[k]):int(batch.struct_ptr[k + 1])] for k in idx}
    parts = run("grad", c, u)
    grad = {name: np.zeros(shape) for name, shape in synth.weight_layout(hp) if not name.startswith("blend")}
    for k in idx:
        for name, val in parts[k].items():
            if name in grad:
                grad[name] += val
    loss_E, loss_F = float(np.mean(np.abs(rE))), float(np.mean(np.abs(rF)))
    return dict(loss=loss_E + force_weight * loss_F, loss_E=loss_E, loss_F=loss_F, E=E, F=Fo, grad=grad)


# The forces pass runs the forward with the filter's bias on the matrix
# cores (the layout its reverse pass reads); the energy-only forward adds it
# in the message epilogue where that saves MFMA work.  Both are checked
# against the oracle; against each other they agree to the precision's
# rounding (relative to the batch's largest energy).
SAME_ENERGY_TOL = {"fp64": 1e-12, "fp32": 1e-5}


def assert_same_energies(E_a, E_b, precision: str, label: str = ""):
    E_a = np.asarray(E_a, dtype=np.float64)
    E_b = np.asarray(E_b, dtype=np.float64)
    assert E_a.shape == E_b.shape, label
    if E_a.size == 0:
        return
    assert np.all(np.isfinite(E_a)) and np.all(np.isfinite(E_b)), label
    scale = max(1.0, float(np.abs(E_b).max()))
    err = float(np.abs(E_a - E_b).max())
    assert err <= SAME_ENERGY_TOL[precision] * scale, f"{label}: forces-pass energies differ by {err:.3e}"
