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
    name, batch_tuple, idx, blend_skip = args
    hp, W = synth.workload_weights(name)
    out = []
    for k, (pos, z, cell, pbc, ds) in zip(idx, batch_tuple):
        if blend_skip is None:
            o = structure_forward(pos, z, cell, pbc, ds if hp.n_heads > 1 else 0, hp, W)
        else:
            o = structure_forward_blend(pos, z, cell, pbc, hp, W, skip=blend_skip)
        out.append((k, o["E"], float(np.sum(np.abs(o["e"])))))
    return out


def _oracle_forces_job(args):
    from oracle.forces import structure_forces
    name, batch_tuple, idx = args
    hp, W = synth.workload_weights(name)
    return [(k, structure_forces(pos, z, cell, pbc, ds if hp.n_heads > 1 else 0, hp, W)["F"])
            for k, (pos, z, cell, pbc, ds) in zip(idx, batch_tuple)]


def oracle_forces(name: str, batch, idx, workers: int | None = None):
    """Oracle forces of structures `idx` of `batch` (list of [n_b, 3]), in a
    process pool."""
    idx = [int(i) for i in idx]
    workers = workers or min(16, os.cpu_count() or 1, max(1, len(idx)))
    chunks = [idx[w::workers] for w in range(workers)]
    jobs = [(name, [batch.structure(k) for k in c], c) for c in chunks if c]
    res = {}
    with ProcessPoolExecutor(workers, initializer=_single_thread_blas) as ex:
        for part in ex.map(_oracle_forces_job, jobs):
            res.update(dict(part))
    return [res[k] for k in idx]


def oracle_energies(name: str, batch, idx, workers: int | None = None, blend_skip=None):
    """Oracle (E, sum|e|) of structures `idx` of `batch`, in a process pool;
    blend_skip given: every head blended, heads below it left out."""
    idx = [int(i) for i in idx]
    workers = workers or min(16, os.cpu_count() or 1, max(1, len(idx)))
    chunks = [idx[w::workers] for w in range(workers)]
    jobs = [(name, [batch.structure(k) for k in c], c, blend_skip) for c in chunks if c]
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


def check_energies(E_gpu, E_ref, A_ref, tol: float, label: str = ""):
    """Assert the tolerance; return (max normalised error, max plain relative error)."""
    E_gpu = np.asarray(E_gpu, dtype=np.float64)
    err = np.abs(E_gpu - E_ref)
    norm = err / A_ref
    rel = err / np.abs(E_ref)
    worst = int(np.argmax(norm))
    assert np.all(np.isfinite(E_gpu)), f"{label}: non-finite energies"
    assert norm.max() <= tol, (f"{label}: max |dE|/sum|e| = {norm.max():.3e} > {tol:.1e} "
                               f"at sample {worst} (E={E_gpu[worst]!r}, ref={E_ref[worst]!r})")
    return float(norm.max()), float(rel.max())
