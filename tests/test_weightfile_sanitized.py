"""The weight-file reader (host code of the C ABI's painn_model_load) built on
its own with AddressSanitizer and UndefinedBehaviorSanitizer, fed valid and
corrupt files: every documented failure gives its status code, no prefix of a
valid file is accepted unless it ends exactly before an optional section, and
no input makes the reader touch memory outside the buffer or hit undefined
behaviour."""
from __future__ import annotations

import os
import shutil
import struct
import subprocess

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_15380_amd", "csrc")
OK, E_FORMAT, E_UNSUPPORTED = 0, -5, -8


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    out = str(tmp_path_factory.mktemp("wf") / "weightfile_check")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(CSRC, "weightfile.cpp"), os.path.join(ROOT, "tests", "native", "weightfile_check.cpp"),
           "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return out


def _run(checker, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([checker, *args], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, f"sanitizer or driver failure:\n{r.stdout}\n{r.stderr}"
    assert "runtime error" not in r.stderr, r.stderr
    return r.stdout


def _small_model(blend=False, cap=0, F=8):
    hp = synth.HyperParams(F=F, K=3, L=1, n_species=3, n_heads=2, cutoff=4.0,
                           shared_dims=[5], branch_dims=[4, 1],
                           blend_dims=[6] if blend else None, max_neighbors=cap)
    return hp, synth.make_weights(hp, 7)


def _header(buf: bytes, **kw) -> bytes:
    """Rewrite header integers of a weight file (F, K, L, n_species, n_heads,
    rbf_type, n_shared, n_branch) or the cutoff."""
    names = ["F", "K", "L", "n_species", "n_heads", "rbf_type", "n_shared", "n_branch"]
    b = bytearray(buf)
    for k, v in kw.items():
        if k == "cutoff":
            struct.pack_into("<d", b, 40, v)
        else:
            struct.pack_into("<i", b, 8 + 4 * names.index(k), v)
    return bytes(b)


def test_reader_statuses(checker, tmp_path):
    hp, W = _small_model(blend=True, cap=5)
    good = synth.weight_file_bytes(hp, W)
    plain = synth.weight_file_bytes(*_small_model())
    hpb, Wb = _small_model(blend=True)
    blend_only = synth.weight_file_bytes(hpb, Wb)
    cap_sec = b"NBRCAP01" + struct.pack("<2i", 5, 0)
    blend_at = blend_only.index(b"BLENDW01")
    blend_sec = blend_only[blend_at:]
    nan_w = bytearray(plain)
    struct.pack_into("<d", nan_w, len(plain) - 8, float("nan"))
    cases = {
        "good": (good, OK),
        "plain": (plain, OK),
        "bad_magic": (b"PAINNW02" + good[8:], E_FORMAT),
        "empty": (b"", E_FORMAT),
        "header_only": (good[:40], E_FORMAT),
        "truncated_arrays": (plain[:-8], E_FORMAT),
        "trailing_zeros": (plain + b"\0" * 8, E_FORMAT),
        "trailing_16": (plain + b"\1" * 16, E_FORMAT),
        "unknown_section": (plain + b"XXXXXXXX" + b"\0" * 8, E_FORMAT),
        "cap_zero": (plain + b"NBRCAP01" + struct.pack("<2i", 0, 0), E_FORMAT),
        "cap_twice": (plain + cap_sec + cap_sec, E_FORMAT),
        "cap_short": (plain + cap_sec[:12], E_FORMAT),
        "blend_twice": (blend_only + blend_sec, E_FORMAT),
        "blend_truncated": (blend_only[:-8], E_FORMAT),
        "blend_bad_count": (blend_only[:blend_at + 8] + struct.pack("<i", 9) + blend_only[blend_at + 12:],
                            E_FORMAT),
        "blend_negative_count": (blend_only[:blend_at + 8] + struct.pack("<i", -1) + blend_only[blend_at + 12:],
                                 E_FORMAT),
        "blend_zero_width": (blend_only[:blend_at + 12] + struct.pack("<i", 0) + blend_only[blend_at + 16:],
                             E_UNSUPPORTED),
        "nan_weight": (bytes(nan_w), E_FORMAT),
        "nan_cutoff": (_header(plain, cutoff=float("nan")), E_FORMAT),
        "neg_cutoff": (_header(plain, cutoff=-1.0), E_FORMAT),
        "F_zero": (_header(plain, F=0), E_UNSUPPORTED),
        "F_385": (_header(plain, F=385), E_UNSUPPORTED),
        "K_one": (_header(plain, K=1), E_UNSUPPORTED),
        "L_zero": (_header(plain, L=0), E_UNSUPPORTED),
        "heads_65": (_header(plain, n_heads=65), E_UNSUPPORTED),
        "rbf_2": (_header(plain, rbf_type=2), E_UNSUPPORTED),
        "species_zero": (_header(plain, n_species=0), E_FORMAT),
        "shared_17": (_header(plain, n_shared=17), E_FORMAT),
        "branch_zero": (_header(plain, n_branch=0), E_FORMAT),
        # header claims more arrays than the file holds
        "L_two": (_header(plain, L=2), E_FORMAT),
    }
    # last branch layer wider than 1: rewrite branch_dims[-1] (after the
    # single shared dim at byte 48 and the first branch dim at 52)
    b = bytearray(plain)
    struct.pack_into("<i", b, 56, 2)
    cases["last_branch_2"] = (bytes(b), E_FORMAT)
    paths = []
    for name, (data, _) in cases.items():
        p = tmp_path / f"{name}.bin"
        p.write_bytes(data)
        paths.append(str(p))
    lines = _run(checker, "one", *paths).splitlines()
    assert len(lines) == len(cases)
    for (name, (_, want)), line in zip(cases.items(), lines):
        st, F, Fl = (int(x) for x in line.split()[:3])
        assert st == want, f"{name}: status {st}, expected {want} ({line})"
        if st == OK:
            assert (F, Fl) == (64, 8), f"{name}: F {F}, F_logical {Fl}"


@pytest.mark.parametrize("blend,cap", [(False, 0), (True, 3)])
def test_reader_rejects_every_prefix(checker, tmp_path, blend, cap):
    """Every prefix fails with PAINN_E_FORMAT except those that end exactly
    where an optional section starts (a complete file without the sections
    after it)."""
    data = synth.weight_file_bytes(*_small_model(blend=blend, cap=cap))
    p = tmp_path / "m.bin"
    p.write_bytes(data)
    ends = []
    for magic in (b"BLENDW01", b"NBRCAP01"):
        if magic in data:
            ends.append(data.index(magic))
    got = [tuple(int(x) for x in l.split()) for l in _run(checker, "prefixes", str(p)).splitlines()]
    assert got == [(n, OK) for n in sorted(ends)]


def test_reader_survives_header_corruption(checker, tmp_path):
    hp, W = _small_model(blend=True, cap=4)
    data = synth.weight_file_bytes(hp, W)
    p = tmp_path / "m.bin"
    p.write_bytes(data)
    out = _run(checker, "flips", str(p), str(len(data)))
    counts = {int(a): int(b) for a, b in (l.split() for l in out.splitlines())}
    assert set(counts) <= {OK, E_FORMAT, E_UNSUPPORTED}, counts
    assert sum(counts.values()) == 3 * len(data)
