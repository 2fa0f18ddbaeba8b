"""ctypes binding of include/painn.h: the same entry points, argument
marshalling only.  Status codes other than PAINN_OK raise PainnError."""
from __future__ import annotations

import ctypes
import os

PAINN_FP64, PAINN_FP32, PAINN_BF16 = 0, 1, 2
PRECISIONS = {"fp64": PAINN_FP64, "fp32": PAINN_FP32, "bf16": PAINN_BF16}

# every symbol declared in include/painn.h
EXPORTS = [
    "painn_create", "painn_set_stream", "painn_destroy", "painn_last_error",
    "painn_status_string", "painn_synchronize", "painn_model_load",
    "painn_model_load_buffer", "painn_model_info", "painn_model_options", "painn_model_free",
    "painn_build_graph", "painn_build_graph_capped", "painn_graph_csr", "painn_graph_free", "painn_forward",
    "painn_forward_noalloc",
    "painn_forward_blend", "painn_forward_features", "painn_forces", "painn_forces_blend",
    "painn_trainer_create", "painn_trainer_step", "painn_trainer_params", "painn_trainer_free",
    "painn_profile_enable",
    "painn_profile_read",
]

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_SIGS = {
    "painn_create": ([ctypes.c_int, _P, ctypes.POINTER(_P)], ctypes.c_int),
    "painn_set_stream": ([_P, _P], ctypes.c_int),
    "painn_destroy": ([_P], ctypes.c_int),
    "painn_last_error": ([_P], ctypes.c_char_p),
    "painn_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "painn_synchronize": ([_P], ctypes.c_int),
    "painn_model_load": ([_P, ctypes.c_char_p, ctypes.POINTER(_P)], ctypes.c_int),
    "painn_model_load_buffer": ([_P, ctypes.c_char_p, ctypes.c_size_t, ctypes.POINTER(_P)], ctypes.c_int),
    "painn_model_info": ([_P] + [ctypes.POINTER(_I32)] * 5 + [ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
    "painn_model_options": ([_P, ctypes.POINTER(_I32), ctypes.POINTER(_I32)], ctypes.c_int),
    "painn_model_free": ([_P], ctypes.c_int),
    "painn_build_graph": ([_P, _I32, _I32, _P, _P, _P, _P, _P, ctypes.c_double, ctypes.POINTER(_P)],
                          ctypes.c_int),
    "painn_build_graph_capped": ([_P, _I32, _I32, _P, _P, _P, _P, _P, ctypes.c_double, _I32,
                                  ctypes.POINTER(_P)], ctypes.c_int),
    "painn_graph_csr": ([_P, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(_I32), ctypes.POINTER(_I32),
                         ctypes.POINTER(_P), ctypes.POINTER(_P), ctypes.POINTER(_P)], ctypes.c_int),
    "painn_graph_free": ([_P], ctypes.c_int),
    "painn_forward": ([_P, _P, _P, _P, ctypes.c_int, _P], ctypes.c_int),
    "painn_forward_noalloc": ([_P, _P, _P, _P, ctypes.c_int, _P], ctypes.c_int),
    "painn_forward_blend": ([_P, _P, _P, ctypes.c_int, ctypes.c_double, _P, _P], ctypes.c_int),
    "painn_forward_features": ([_P, _P, _P, ctypes.c_int, _I32, _P, _P], ctypes.c_int),
    "painn_forces": ([_P, _P, _P, _P, ctypes.c_int, _P, _P], ctypes.c_int),
    "painn_forces_blend": ([_P, _P, _P, ctypes.c_int, ctypes.c_double, _P, _P, _P], ctypes.c_int),
    "painn_trainer_create": ([_P, _P, _P, ctypes.POINTER(_P)], ctypes.c_int),
    "painn_trainer_step": ([_P, _P, _P, _P, _P, _P], ctypes.c_int),
    "painn_trainer_params": ([_P, ctypes.POINTER(ctypes.c_int64), _P, _P], ctypes.c_int),
    "painn_trainer_free": ([_P], ctypes.c_int),
    "painn_profile_enable": ([_P, ctypes.c_int], ctypes.c_int),
    "painn_profile_read": ([_P, _I32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_double),
                            ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(_I32)], ctypes.c_int),
}

_LIB = None


def lib_path() -> str:
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpainn.so")


def load_library():
    """Load libpainn.so (built by paper_2604_15380_amd.build); raises if absent."""
    global _LIB
    if _LIB is None:
        p = lib_path()
        if not os.path.exists(p):
            raise RuntimeError(f"{p} is not built: run paper_2604_15380_amd.build.build() "
                               "(there is no fallback path)")
        lib = ctypes.CDLL(p)
        for name, (args, res) in _SIGS.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        _LIB = lib
    return _LIB


class PainnError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        super().__init__(f"{painn_status_string(status)}: {message}")


def _check(st: int, ctx=None):
    if st != 0:
        msg = load_library().painn_last_error(ctx).decode() if ctx else ""
        raise PainnError(st, msg)


def painn_status_string(status: int) -> str:
    return load_library().painn_status_string(status).decode()


def painn_create(device: int, stream: int | None) -> int:
    out = _P()
    st = load_library().painn_create(device, stream or None, ctypes.byref(out))
    if st != 0:
        raise PainnError(st, f"cannot create a context on device {device}")
    return out.value


def painn_set_stream(ctx: int, stream: int | None) -> None:
    _check(load_library().painn_set_stream(ctx, stream or None), ctx)


def painn_destroy(ctx: int) -> None:
    _check(load_library().painn_destroy(ctx))


def painn_last_error(ctx: int) -> str:
    return load_library().painn_last_error(ctx).decode()


def painn_synchronize(ctx: int) -> None:
    _check(load_library().painn_synchronize(ctx), ctx)


def painn_model_load(ctx: int, path: str) -> int:
    out = _P()
    _check(load_library().painn_model_load(ctx, path.encode(), ctypes.byref(out)), ctx)
    return out.value


def painn_model_load_buffer(ctx: int, data: bytes) -> int:
    out = _P()
    _check(load_library().painn_model_load_buffer(ctx, data, len(data), ctypes.byref(out)), ctx)
    return out.value


def painn_model_info(model: int) -> dict:
    v = [_I32() for _ in range(5)]
    rc = ctypes.c_double()
    _check(load_library().painn_model_info(model, *[ctypes.byref(x) for x in v], ctypes.byref(rc)))
    return dict(F=v[0].value, K=v[1].value, L=v[2].value, n_species=v[3].value,
                n_heads=v[4].value, cutoff=rc.value)


def painn_model_options(model: int) -> dict:
    hb, mn = _I32(), _I32()
    _check(load_library().painn_model_options(model, ctypes.byref(hb), ctypes.byref(mn)))
    return dict(has_blend=bool(hb.value), max_neighbors=mn.value)


def painn_model_free(model: int) -> None:
    _check(load_library().painn_model_free(model))


def painn_build_graph(ctx: int, n_struct: int, n_atoms: int, struct_ptr: int, pos: int,
                      species: int, cell: int | None, pbc: int | None, cutoff: float,
                      graph: int | None = None) -> int:
    g = _P(graph)
    _check(load_library().painn_build_graph(ctx, n_struct, n_atoms, struct_ptr, pos, species,
                                            cell or None, pbc or None, cutoff, ctypes.byref(g)), ctx)
    return g.value


def painn_build_graph_capped(ctx: int, n_struct: int, n_atoms: int, struct_ptr: int, pos: int,
                             species: int, cell: int | None, pbc: int | None, cutoff: float,
                             max_neighbors: int, graph: int | None = None) -> int:
    g = _P(graph)
    _check(load_library().painn_build_graph_capped(ctx, n_struct, n_atoms, struct_ptr, pos, species,
                                                   cell or None, pbc or None, cutoff, max_neighbors,
                                                   ctypes.byref(g)), ctx)
    return g.value


def painn_graph_csr(graph: int) -> dict:
    ne = ctypes.c_int64()
    na, nb = _I32(), _I32()
    rp, col, sh = _P(), _P(), _P()
    _check(load_library().painn_graph_csr(graph, ctypes.byref(ne), ctypes.byref(na), ctypes.byref(nb),
                                          ctypes.byref(rp), ctypes.byref(col), ctypes.byref(sh)))
    return dict(n_edges=ne.value, n_atoms=na.value, n_struct=nb.value, row_ptr=rp.value,
                col=col.value, shift=sh.value)


def painn_graph_free(graph: int) -> None:
    _check(load_library().painn_graph_free(graph))


def painn_forward(ctx: int, model: int, graph: int, dataset_id: int | None, precision: int,
                  energies: int) -> None:
    _check(load_library().painn_forward(ctx, model, graph, dataset_id or None, precision, energies), ctx)


def painn_forward_noalloc(ctx: int, model: int, graph: int, dataset_id: int | None, precision: int,
                          energies: int) -> None:
    _check(load_library().painn_forward_noalloc(ctx, model, graph, dataset_id or None, precision, energies),
           ctx)


def painn_forward_blend(ctx: int, model: int, graph: int, precision: int, skip_threshold: float,
                        energies: int, weights: int | None) -> None:
    _check(load_library().painn_forward_blend(ctx, model, graph, precision, float(skip_threshold),
                                              energies, weights or None), ctx)


def painn_forces(ctx: int, model: int, graph: int, dataset_id: int | None, precision: int,
                 energies: int | None, forces: int | None) -> None:
    _check(load_library().painn_forces(ctx, model, graph, dataset_id or None, precision,
                                       energies or None, forces or None), ctx)


def painn_forces_blend(ctx: int, model: int, graph: int, precision: int, skip_threshold: float,
                       energies: int | None, forces: int | None, weights: int | None) -> None:
    _check(load_library().painn_forces_blend(ctx, model, graph, precision, float(skip_threshold),
                                             energies or None, forces or None, weights or None), ctx)


def painn_forward_features(ctx: int, model: int, graph: int, precision: int, layer: int,
                           s_out: int, v_out: int) -> None:
    _check(load_library().painn_forward_features(ctx, model, graph, precision, layer, s_out, v_out), ctx)


class painn_train_config(ctypes.Structure):
    """include/painn.h painn_train_config (host struct)."""
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double), ("force_weight", ctypes.c_double)]


def painn_trainer_create(ctx: int, model: int, cfg: dict | None = None) -> int:
    out = _P()
    c = None
    if cfg is not None:
        c = painn_train_config(**cfg)
    _check(load_library().painn_trainer_create(ctx, model, ctypes.addressof(c) if c is not None else None,
                                               ctypes.byref(out)), ctx)
    return out.value


def painn_trainer_step(ctx: int, trainer: int, graph: int, dataset_id: int | None, energy_ref: int | None,
                       force_ref: int | None, loss: int | None) -> None:
    _check(load_library().painn_trainer_step(trainer, graph, dataset_id or None, energy_ref or None,
                                             force_ref or None, loss or None), ctx)


def painn_trainer_params(ctx: int, trainer: int, params: int | None = None, grad: int | None = None) -> int:
    n = ctypes.c_int64()
    _check(load_library().painn_trainer_params(trainer, ctypes.byref(n), params or None, grad or None), ctx)
    return n.value


def painn_trainer_free(trainer: int) -> None:
    _check(load_library().painn_trainer_free(trainer))


def painn_profile_enable(ctx: int, enable: bool) -> None:
    _check(load_library().painn_profile_enable(ctx, 1 if enable else 0), ctx)


def painn_profile_read(ctx: int) -> dict:
    """{kernel class: (milliseconds, launches)} accumulated since the last read."""
    n_max = 32
    names = (ctypes.c_char_p * n_max)()
    ms = (ctypes.c_double * n_max)()
    cnt = (ctypes.c_int64 * n_max)()
    n = _I32()
    _check(load_library().painn_profile_read(ctx, n_max, names, ms, cnt, ctypes.byref(n)), ctx)
    return {names[k].decode(): (ms[k], cnt[k]) for k in range(n.value)}
