"""CPU checks of the boundary: the built library exports every entry point
declared in include/painn.h, the binding covers exactly those, and the host
logic that needs no device (status names, the weight-file format) works."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2604_15380_amd as pk
from paper_2604_15380_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "painn.h")


def header_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(painn_[a-z_]+)\s*\(", txt)))


def test_header_declares_the_binding_exports():
    assert header_functions() == sorted(binding.EXPORTS)


@pytest.mark.skipif(not os.path.exists(binding.lib_path()), reason="library not built")
def test_library_exports_every_header_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", binding.lib_path()],
                         capture_output=True, text=True, check=True).stdout
    syms = {l.split()[-1] for l in out.splitlines() if l.strip()}
    for fn in header_functions():
        assert fn in syms, fn
    lib = ctypes.CDLL(binding.lib_path())
    for fn in header_functions():
        assert getattr(lib, fn) is not None


@pytest.mark.skipif(not os.path.exists(binding.lib_path()), reason="library not built")
def test_status_strings_without_device():
    assert pk.painn_status_string(0) == "PAINN_OK"
    assert pk.painn_status_string(-7) == "PAINN_E_COINCIDENT"
    assert pk.painn_status_string(-99) == "PAINN_E_UNKNOWN"


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(binding, "_LIB", None)
    monkeypatch.setattr(binding, "lib_path", lambda: str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        binding.load_library()


@pytest.mark.skipif(not os.path.exists(binding.lib_path()), reason="library not built")
def test_null_handles_without_device():
    """Every entry point given a null context or null handle returns its
    documented status (PAINN_E_ARG; PAINN_OK for the *_free calls and
    painn_destroy) before any device call, so this runs without a GPU."""
    lib = binding.load_library()
    E_ARG = -1
    out = ctypes.c_void_p()
    i32 = ctypes.c_int32()
    d = ctypes.c_double()
    i64 = ctypes.c_int64()
    names = (ctypes.c_char_p * 4)()
    ms = (ctypes.c_double * 4)()
    cnt = (ctypes.c_int64 * 4)()
    r = ctypes.byref
    assert lib.painn_create(0, None, None) == E_ARG
    assert lib.painn_set_stream(None, None) == E_ARG
    assert lib.painn_destroy(None) == 0
    assert lib.painn_last_error(None) == b"null context"
    assert lib.painn_synchronize(None) == E_ARG
    assert lib.painn_model_load(None, b"/nonexistent", r(out)) == E_ARG
    assert lib.painn_model_load_buffer(None, b"PAINNW01", 8, r(out)) == E_ARG
    assert lib.painn_model_info(None, r(i32), r(i32), r(i32), r(i32), r(i32), r(d)) == E_ARG
    assert lib.painn_model_options(None, r(i32), r(i32)) == E_ARG
    assert lib.painn_model_free(None) == 0
    assert lib.painn_build_graph(None, 1, 1, None, None, None, None, None, 5.0, r(out)) == E_ARG
    assert lib.painn_build_graph_capped(None, 1, 1, None, None, None, None, None, 5.0, 3, r(out)) == E_ARG
    assert lib.painn_graph_csr(None, r(i64), r(i32), r(i32), None, None, None) == E_ARG
    assert lib.painn_graph_free(None) == 0
    assert lib.painn_forward(None, None, None, None, 0, None) == E_ARG
    assert lib.painn_forward_blend(None, None, None, 0, 0.0, None, None) == E_ARG
    assert lib.painn_forward_features(None, None, None, 0, 0, None, None) == E_ARG
    assert lib.painn_forces(None, None, None, None, 0, None, None) == E_ARG
    assert lib.painn_forces_blend(None, None, None, 0, 0.0, None, None, None) == E_ARG
    assert lib.painn_forward_noalloc(None, None, None, None, 0, None) == E_ARG
    assert lib.painn_trainer_create(None, None, None, r(out)) == E_ARG
    assert lib.painn_trainer_step(None, None, None, None, None, None) == E_ARG
    assert lib.painn_trainer_params(None, r(i64), None, None) == E_ARG
    assert lib.painn_trainer_free(None) == 0
    assert lib.painn_profile_enable(None, 1) == E_ARG
    assert lib.painn_profile_read(None, 4, names, ms, cnt, r(i32)) == E_ARG
