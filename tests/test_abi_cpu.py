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
